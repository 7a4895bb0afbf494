// Mixer epilogue (Sec. 3.4): head coupling, sigmoid gate and causal depthwise
// local path around the resonant mixing output.
//
//   C = I + (lambda_c / sqrt(H)) tanh(Ct)                       coupling eq.
//   ybar[b,t,g dh + j] = sum_h C[g,h] y[b,t,h dh + j]           head mixing eq.
//   l[b,t,c] = sum_{k<K} w[c,k] v[b,t-k,c]   (zero before t = 0)  local path
//   z = sigmoid(gate) * ybar + s * l                            combine eq.
//
// The kernels are meant to be bound by HBM traffic: every activation element is
// read once from HBM.  Forward: a thread owns a piece of adjacent channels at
// the same position j of every head (epi_fwd_col_kernel), so the head mixing
// needs no other thread's data; the K-1 earlier rows of the local path are
// neighbouring threads' rows and hit in cache.  Backward: row chunks are staged
// in LDS (epi_bwd_tile_kernel), since dy at one head needs dz sigmoid(gate) of
// every head.  Shapes outside those kernels' limits take the generic kernels
// below (one piece of VEC channels of one head per thread).
//
// Backward (loss sum(dz z)), with sg = sigmoid(gate), dyb = dz sg, dl = dz s:
//   dgate = dz ybar sg (1 - sg);  dy[h dh + j] = sum_g C[g,h] dyb[g dh + j];
//   dv[t] = sum_k w[k] dl[t+k];   and the parameter sums over (b, t)
//   dC[g,h] = sum dyb[g dh + j] y[h dh + j],  ds = sum dz l,  dw[k] = sum dl[t] v[t-k],
// reduced per block of rows (float32, fixed order), then over blocks (float64,
// fixed order), so they are bitwise reproducible.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "proj.h"

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
// with the hardware reciprocal (about 1 ulp), for the tile kernels
__device__ __forceinline__ float sigmoid_fast(float u) { return __builtin_amdgcn_rcpf(1.f + __expf(-u)); }

// C = I + (lambda_c / sqrt(H)) tanh(Ct) into LDS (all threads; the caller syncs)
__device__ __forceinline__ void coupling_to_lds(float* sC, const float* Ct, float lambda_c, int H) {
  const float scale = lambda_c / sqrtf((float)H);
  for (int i = threadIdx.x; i < H * H; i += blockDim.x)
    sC[i] = (i / H == i % H ? 1.f : 0.f) + scale * tanhf(Ct[i]);
}

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
  // partials are stored column-major: entry e of this block at part[e * gridDim.x + blockIdx.x]
  auto out = [&](int e) -> float& { return part[(size_t)e * gridDim.x + blockIdx.x]; };
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
        out(H * H + c) = ds;
#pragma unroll
        for (int k = 0; k < EPI_K_MAX; ++k)
          if (k < K) out(H * H + D + c * K + k) = dw[k];
      }
    }
    // dC[g, h] += sum over this channel block's channels of head g, in order
#pragma unroll
    for (int h = 0; h < EPI_H_MAX; ++h)
      if (h < H) sdc[threadIdx.x * EPI_H_MAX + h] = live ? dc[h] : 0.f;
    __syncthreads();
    for (int e = threadIdx.x; e < H * H; e += blockDim.x) {
      const int gg = e / H, h = e % H;
      float acc = cb == 0 ? 0.f : out(e);
      for (int q = 0; q < (int)blockDim.x; ++q) {
        const int cc = cb + q;
        if (cc < D && cc / dh == gg) acc += sdc[q * EPI_H_MAX + h];
      }
      out(e) = acc;
    }
    __syncthreads();
  }
}

// Sum of the block partials in float64, in a fixed order, then the chain rule of
// the coupling map.  A block takes 16 partial columns; its 16 row groups each sum
// every 16th block partial (two interleaved accumulators), and the row groups
// are added in order.
// One wave per partial column (the partials are column-major, so a column is
// contiguous): lane l sums partial rows l, l + 64, ... in float64 with four
// accumulators in a fixed order, then the lane sums meet in a fixed shuffle tree.
__global__ __launch_bounds__(256) void epi_bwd_reduce_kernel(const float* __restrict__ part, int64_t nparts, int H,
                                                             int D, int K, const float* __restrict__ Ct,
                                                             float lambda_c, float* __restrict__ dCt,
                                                             float* __restrict__ dw, float* __restrict__ ds,
                                                             double* __restrict__ lam_terms) {
  const int P = H * H + D + D * K;
  const int lane = threadIdx.x & 63, col = blockIdx.x * 4 + threadIdx.x / 64;
  if (col >= P) return;  // the whole wave: no barrier follows
  const float* pc = part + (size_t)col * nparts;
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
  int64_t k = lane;
  for (; k + 192 < nparts; k += 256) {
    a0 += pc[k];
    a1 += pc[k + 64];
    a2 += pc[k + 128];
    a3 += pc[k + 192];
  }
  for (; k < nparts; k += 64) a0 += pc[k];
  double acc = (a0 + a1) + (a2 + a3);
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_down(acc, off, 64);
  if (lane != 0) return;
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

// dlambda_c = sum_{g,h} dC[g,h] tanh(Ct[g,h]) / sqrt(H), one wave, fixed order
__global__ __launch_bounds__(64) void epi_bwd_lambda_kernel(const double* __restrict__ lam_terms, int H,
                                                            float* __restrict__ dlambda_c) {
  double u = 0.0;
  for (int i = threadIdx.x; i < H * H; i += 64) u += lam_terms[i];
  for (int off = 32; off > 0; off >>= 1) u += __shfl_down(u, off, 64);
  if (threadIdx.x == 0) *dlambda_c = (float)(u / sqrt((double)H));
}

// ---------------------------------------------------------------------------
// Tile kernels.  A block works on chunks of R consecutive rows of one batch
// row.  A thread owns one piece of CPT adjacent channels (a 16-byte vector in
// the forward, an 8-byte one in the backward, or one element when the heads or
// pointers do not allow that) in every RP-th row of the chunk: thread (rr, cg)
// has piece cg of rows rr, rr + RP, ...  Every activation row window a chunk
// needs (its own rows; the K-1 rows before it for the local path, after it for
// dv) is copied to LDS with one pass of vector loads issued before any LDS
// store, so the head sums and the taps read LDS.  In the backward a thread's
// piece is the same in every chunk, so the parameter sums (dC, ds, dw) stay in
// registers across all chunks the block takes, and each block writes one
// partial row [H*H dC | D ds | D*K dw] at the end.
// ---------------------------------------------------------------------------
template <int N> struct U32V { typedef uint32_t type __attribute__((ext_vector_type(N))); };
template <int N> struct F32V { typedef float type __attribute__((ext_vector_type(N))); };

// A piece: raw = the activation bits moved by one load or store, fraw = a
// float32 copy kept in LDS.
template <typename T, int CPT> struct Pc;
template <int CPT> struct Pc<bf16_t, CPT> {
  typedef typename U32V<CPT / 2>::type raw;
  typedef typename F32V<CPT>::type fraw;
  __device__ static void unpack(raw r, float (&f)[CPT]) {
#pragma unroll
    for (int i = 0; i < CPT / 2; ++i)
      f[2 * i] = __uint_as_float(r[i] << 16), f[2 * i + 1] = __uint_as_float(r[i] & 0xFFFF0000u);
  }
  __device__ static raw pack(const float (&f)[CPT]) {
    raw r;
#pragma unroll
    for (int i = 0; i < CPT / 2; ++i)
      r[i] = (uint32_t)from_f32<bf16_t>(f[2 * i]) | ((uint32_t)from_f32<bf16_t>(f[2 * i + 1]) << 16);
    return r;
  }
};
template <int CPT> struct Pc<float, CPT> {
  typedef typename U32V<CPT>::type raw;
  typedef typename F32V<CPT>::type fraw;
  __device__ static void unpack(raw r, float (&f)[CPT]) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) f[i] = __uint_as_float(r[i]);
  }
  __device__ static raw pack(const float (&f)[CPT]) {
    raw r;
#pragma unroll
    for (int i = 0; i < CPT; ++i) r[i] = __float_as_uint(f[i]);
    return r;
  }
};
template <> struct Pc<bf16_t, 1> {
  typedef bf16_t raw;
  typedef float fraw;
  __device__ static void unpack(raw r, float (&f)[1]) { f[0] = to_f32(r); }
  __device__ static raw pack(const float (&f)[1]) { return from_f32<bf16_t>(f[0]); }
};
template <> struct Pc<float, 1> {
  typedef float raw;
  typedef float fraw;
  __device__ static void unpack(raw r, float (&f)[1]) { f[0] = r; }
  __device__ static raw pack(const float (&f)[1]) { return f[0]; }
};
template <int CPT> __device__ __forceinline__ void funpack(typename F32V<CPT>::type r, float (&f)[CPT]) {
#pragma unroll
  for (int i = 0; i < CPT; ++i) f[i] = r[i];
}
__device__ __forceinline__ void funpack(float r, float (&f)[1]) { f[0] = r; }
template <int CPT> __device__ __forceinline__ typename F32V<CPT>::type fpack(const float (&f)[CPT]) {
  typename F32V<CPT>::type r;
#pragma unroll
  for (int i = 0; i < CPT; ++i) r[i] = f[i];
  return r;
}
__device__ __forceinline__ float fpack(const float (&f)[1]) { return f[0]; }

// channels per piece: 16 bytes forward, 8 bytes backward (register budget)
template <typename T> constexpr int tile_wide(bool bwd) { return (bwd ? 8 : 16) / (int)sizeof(T); }
constexpr int tile_kmax(int cpt) { return cpt > 1 ? 4 : EPI_K_MAX; }

struct TileGeo {
  int D, G, RP;  // channels, pieces per row, rows per pass (threads G * RP)
};
__host__ __device__ inline TileGeo tile_geo(int D, int cpt) {
  TileGeo t;
  t.D = D, t.G = D / cpt, t.RP = 256 / t.G;
  return t;
}

// Forward, one thread per (row, column piece): the thread owns channels
// j0 .. j0+CPT-1 of every head in one row, so it loads each y and gate element
// of its piece exactly once and forms all H mixed heads from them in registers
// (H*H*CPT multiply-adds).  The local path reads v at the K-1 previous rows too;
// those are the current rows of neighbouring threads, so they hit in cache.  No
// LDS staging, no barriers after the prologue: every load of a row is issued
// before any of it is used.
template <typename T, int CPT, int HM, bool WL>
__global__ __launch_bounds__(256) void epi_fwd_col_kernel(const T* __restrict__ y, const T* __restrict__ gate,
                                                          const T* __restrict__ v, T* __restrict__ z,
                                                          int64_t rows, int64_t L, int H, int dh, int K,
                                                          const float* __restrict__ Ct, float lambda_c,
                                                          const float* __restrict__ w,
                                                          const float* __restrict__ s) {
  typedef Pc<T, CPT> PC;
  typedef typename PC::raw P;
  __shared__ float sC[EPI_H_MAX * EPI_H_MAX];
  extern __shared__ __align__(16) float sW[];  // w as [K][D], then s[D] (WL: taps in LDS)
  coupling_to_lds(sC, Ct, lambda_c, H);
  const int D = H * dh, np = dh / CPT;
  if (WL) {
    for (int x = threadIdx.x; x < D * K; x += blockDim.x) sW[(x % K) * D + x / K] = w[x];
    if (K > 0)
      for (int x = threadIdx.x; x < D; x += blockDim.x) sW[D * K + x] = s[x];
  }
  __syncthreads();
  // A block step covers RB rows x PB pieces (PB = min(np, 256)); the row and its
  // position in the batch row come from block-uniform (scalar) arithmetic.
  const int PB = np < (int)blockDim.x ? np : (int)blockDim.x, RB = (int)blockDim.x / PB;
  const int rl = (int)threadIdx.x / PB, pl = (int)threadIdx.x - rl * PB;
  const int64_t ncb = (np + PB - 1) / PB, nq = (rows + RB - 1) / RB * ncb;
  if (rl >= RB) return;  // no barrier follows
  for (int64_t q = blockIdx.x; q < nq; q += gridDim.x) {
    const int64_t rb = q / ncb * RB;
    const int p = (int)(q % ncb) * PB + pl;
    const int64_t r = rb + rl;
    if (r >= rows || p >= np) continue;
    int64_t t = rb % L + rl;
    while (t >= L) t -= L;  // the step's rows may cross into the next batch row
    const int j0 = p * CPT;
    const int64_t o = r * D + j0;
    if constexpr (HM == 8 && CPT > 1) {
      // Every load of the row is issued before any is used: a head at or beyond
      // H, a tap at or beyond K and a tap before t = 0 read a valid row of this
      // batch row and get a zero weight, so no load waits behind a branch.  v is
      // read only when K > 0 (it may be null otherwise); that branch is uniform.
      P yr[8], gr[8], vr[8][4];
#pragma unroll
      for (int h = 0; h < 8; ++h) {
        const int hh = h < H ? h : 0;
        yr[h] = *reinterpret_cast<const P*>(y + o + hh * dh);
        gr[h] = *reinterpret_cast<const P*>(gate + o + hh * dh);
      }
      if (K > 0) {
#pragma unroll
        for (int h = 0; h < 8; ++h) {
          const int hh = h < H ? h : 0;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const bool tap = k < K && k <= t;  // then row r - k is in this batch row
            vr[h][k] = *reinterpret_cast<const P*>(v + o - (tap ? (int64_t)k * D : 0) + hh * dh);
          }
        }
      }
      float acc[8][CPT];
#pragma unroll
      for (int g = 0; g < 8; ++g)
#pragma unroll
        for (int e = 0; e < CPT; ++e) acc[g][e] = 0.f;
#pragma unroll
      for (int h = 0; h < 8; ++h) {
        float yh[CPT];
        PC::unpack(yr[h], yh);
#pragma unroll
        for (int g = 0; g < 8; ++g) {
          const float cgh = (g < H && h < H) ? sC[g * H + h] : 0.f;
#pragma unroll
          for (int e = 0; e < CPT; ++e) acc[g][e] = fmaf(cgh, yh[e], acc[g][e]);
        }
      }
#pragma unroll
      for (int g = 0; g < 8; ++g) {
        if (g >= H) continue;
        const int c0 = g * dh + j0;
        float u[CPT], out[CPT], l[CPT];
        PC::unpack(gr[g], u);
#pragma unroll
        for (int e = 0; e < CPT; ++e) out[e] = sigmoid_fast(u[e]) * acc[g][e], l[e] = 0.f;
        if (K > 0) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const bool tap = k < K && k <= t;
            float vv[CPT];
            PC::unpack(vr[g][k], vv);
#pragma unroll
            for (int e = 0; e < CPT; ++e)
              l[e] = fmaf(tap ? (WL ? sW[k * D + c0 + e] : w[(c0 + e) * K + k]) : 0.f, vv[e], l[e]);
          }
#pragma unroll
          for (int e = 0; e < CPT; ++e) out[e] = fmaf(WL ? sW[D * K + c0 + e] : s[c0 + e], l[e], out[e]);
        }
        *reinterpret_cast<P*>(z + o + g * dh) = PC::pack(out);
      }
    } else {
      float acc[HM][CPT];
#pragma unroll
      for (int g = 0; g < HM; ++g)
#pragma unroll
        for (int e = 0; e < CPT; ++e) acc[g][e] = 0.f;
#pragma unroll
      for (int h = 0; h < HM; ++h) {
        if (h < H) {
          float yh[CPT];
          PC::unpack(*reinterpret_cast<const P*>(y + o + h * dh), yh);
#pragma unroll
          for (int g = 0; g < HM; ++g) {
            if (g < H) {
              const float cgh = sC[g * H + h];
#pragma unroll
              for (int e = 0; e < CPT; ++e) acc[g][e] = fmaf(cgh, yh[e], acc[g][e]);
            }
          }
        }
      }
#pragma unroll
      for (int g = 0; g < HM; ++g) {
        if (g < H) {
          const int c0 = g * dh + j0;
          float u[CPT], out[CPT];
          PC::unpack(*reinterpret_cast<const P*>(gate + o + g * dh), u);
#pragma unroll
          for (int e = 0; e < CPT; ++e) out[e] = sigmoid_fast(u[e]) * acc[g][e];
          if (K > 0) {
            float l[CPT];
#pragma unroll
            for (int e = 0; e < CPT; ++e) l[e] = 0.f;
            for (int k = 0; k < K && k <= t; ++k) {
              float vv[CPT];
              PC::unpack(*reinterpret_cast<const P*>(v + o - (int64_t)k * D + g * dh), vv);
#pragma unroll
              for (int e = 0; e < CPT; ++e)
                l[e] = fmaf(WL ? sW[k * D + c0 + e] : w[(c0 + e) * K + k], vv[e], l[e]);
            }
#pragma unroll
            for (int e = 0; e < CPT; ++e) out[e] = fmaf(WL ? sW[D * K + c0 + e] : s[c0 + e], l[e], out[e]);
          }
          *reinterpret_cast<P*>(z + o + g * dh) = PC::pack(out);
        }
      }
    }
  }
}

// Row windows of a chunk: rows t_first .. t_first + nrows - 1 of batch row b,
// zero outside [0, L).  Thread (rr, cg) moves piece cg of window rows rr + u RP,
// u < U; the host keeps every window within U RP rows.  Loads for the next
// chunk are issued into registers before the current chunk is computed, and
// written to LDS (as float32, the gate as it is) after it.
struct WinSrc {
  int64_t t_first;
  int nrows;
};

template <typename T, int CPT, int U, int NW>
__device__ __forceinline__ void win_load(typename Pc<T, CPT>::raw (&r)[NW][U], const T* const (&src)[NW],
                                         const WinSrc (&w)[NW], int64_t b, int64_t L, int D, int rr, int cg,
                                         int RP) {
  typedef typename Pc<T, CPT>::raw P;
#pragma unroll
  for (int q = 0; q < NW; ++q)
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = rr + u * RP;
      const int64_t t = w[q].t_first + i;
      if (i < w[q].nrows && t >= 0 && t < L)
        r[q][u] = *reinterpret_cast<const P*>(src[q] + (b * L + t) * D + cg * CPT);
      else
        r[q][u] = P(0);
    }
}

// window 0 (the gate) is stored as it is, windows 1.. as float32
template <typename T, int CPT, int U, int NW>
__device__ __forceinline__ void win_store(const typename Pc<T, CPT>::raw (&r)[NW][U],
                                          typename Pc<T, CPT>::raw* gdst,
                                          typename Pc<T, CPT>::fraw* const (&fdst)[NW - 1], const WinSrc (&w)[NW],
                                          int G, int rr, int cg, int RP) {
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (rr + u * RP < w[0].nrows) gdst[(rr + u * RP) * G + cg] = r[0][u];
#pragma unroll
  for (int q = 1; q < NW; ++q)
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (rr + u * RP < w[q].nrows) {
        float f[CPT];
        Pc<T, CPT>::unpack(r[q][u], f);
        fdst[q - 1][(rr + u * RP) * G + cg] = fpack(f);
      }
}

// The backward's windows into LDS as loaded (the element type; unpacked to
// float32 where they are read, which is exact).
template <typename T, int CPT, int U, int NW>
__device__ __forceinline__ void win_store_raw(const typename Pc<T, CPT>::raw (&r)[NW][U],
                                              typename Pc<T, CPT>::raw* const (&dst)[NW], const WinSrc (&w)[NW],
                                              int G, int rr, int cg, int RP) {
#pragma unroll
  for (int q = 0; q < NW; ++q)
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (rr + u * RP < w[q].nrows) dst[q][(rr + u * RP) * G + cg] = r[q][u];
}

// Per-thread local-path parameters, read once before the chunk loop.  They go
// through LDS: the compiler waits for every outstanding global load before a
// loop that stores but does not load whenever that loop uses a register
// loaded from global memory, which would stall on the next chunk's prefetch.
template <int CPT, int KM>
__device__ __forceinline__ void params_via_lds(float (&wk)[KM][CPT], float (&sc)[CPT], const float* w,
                                               const float* s, int D, int K, int c0, bool act, float* sp) {
  for (int x = threadIdx.x; x < D * K; x += blockDim.x) sp[x] = w[x];
  if (K > 0)
    for (int x = threadIdx.x; x < D; x += blockDim.x) sp[D * K + x] = s[x];
  __syncthreads();
#pragma unroll
  for (int e = 0; e < CPT; ++e) {
    sc[e] = (act && K > 0) ? sp[D * K + c0 + e] : 0.f;
#pragma unroll
    for (int k = 0; k < KM; ++k) wk[k][e] = (act && k < K) ? sp[(c0 + e) * K + k] : 0.f;
  }
  __syncthreads();  // the area is reused for the row windows
}

// rows of one window slot per thread: the forward moves 3 windows, the backward 4
template <int CPT> constexpr int tile_u(bool bwd) { return CPT == 1 ? 16 : (bwd ? 5 : 3); }

template <typename T, int CPT, int HM>
__global__ __launch_bounds__(256) void epi_bwd_tile_kernel(const T* __restrict__ y, const T* __restrict__ gate,
                                                           const T* __restrict__ v, const T* __restrict__ dz,
                                                           T* __restrict__ dy, T* __restrict__ dgate,
                                                           T* __restrict__ dv, int64_t B, int64_t L, int H, int dh,
                                                           int K, int R, const float* __restrict__ Ct,
                                                           float lambda_c, const float* __restrict__ w,
                                                           const float* __restrict__ s, float* __restrict__ part) {
  typedef Pc<T, CPT> PC;
  typedef typename PC::raw P;
  typedef typename PC::fraw PF;
  constexpr int KM = tile_kmax(CPT), U = tile_u<CPT>(true);
  __shared__ float sC[EPI_H_MAX * EPI_H_MAX];
  extern __shared__ __align__(16) unsigned char smem[];
  const TileGeo tg = tile_geo(H * dh, CPT);
  const int D = tg.D, G = tg.G, RP = tg.RP, KH = K > 0 ? K - 1 : 0;
  PF* dybs = reinterpret_cast<PF*>(smem);  // [R][G]  dz sigmoid(gate), float32
  P* ys = reinterpret_cast<P*>(dybs + R * G);  // [R][G]; the windows as loaded
  P* dzs = ys + R * G;                     // [R + KH][G]: rows t0 .. t0 + R + KH - 1
  P* vs = dzs + (R + KH) * G;              // [R + KH][G]: rows t0 - KH .. t0 + R - 1
  P* gs = vs + (K > 0 ? R + KH : 0) * G;   // [R][G] gate
  coupling_to_lds(sC, Ct, lambda_c, H);
  const int rr = threadIdx.x / G, cg = threadIdx.x % G;
  const bool act = rr < RP;
  const int c0 = cg * CPT, g = c0 / dh, j0 = c0 % dh;
  float wk[KM][CPT], sc[CPT], dw[KM][CPT], ds[CPT], dc[HM];
  params_via_lds<CPT, KM>(wk, sc, w, s, D, K, c0, act, reinterpret_cast<float*>(smem));
#pragma unroll
  for (int e = 0; e < CPT; ++e) {
    ds[e] = 0.f;
#pragma unroll
    for (int k = 0; k < KM; ++k) dw[k][e] = 0.f;
  }
#pragma unroll
  for (int h = 0; h < HM; ++h) dc[h] = 0.f;
  const int64_t nct = (L + R - 1) / R, nch = B * nct;
  const T* const src[4] = {gate, y, dz, v};
  P* const wdst[4] = {gs, ys, dzs, vs};
  auto wins = [&](int64_t c, WinSrc (&wv)[4]) {
    const int64_t t0 = (c % nct) * R;
    const int n = (int)(L - t0 < R ? L - t0 : R);
    wv[0] = {t0, n}, wv[1] = {t0, n}, wv[2] = {t0, n + KH}, wv[3] = {t0 - KH, K > 0 ? n + KH : 0};
  };
  P r[4][U];
  WinSrc wv[4];
  int64_t c = blockIdx.x;
  if (act && c < nch) {
    wins(c, wv);
    win_load<T, CPT, U, 4>(r, src, wv, c / nct, L, D, rr, cg, RP);
  }
  for (; c < nch; c += gridDim.x) {
    const int64_t b = c / nct, t0 = (c % nct) * R;
    const int n = (int)(L - t0 < R ? L - t0 : R);
    __syncthreads();
    if (act) {
      wins(c, wv);
      win_store_raw<T, CPT, U, 4>(r, wdst, wv, G, rr, cg, RP);
      for (int i = rr; i < n; i += RP) {  // own pieces, just stored by this thread
        float u[CPT], zz[CPT], db[CPT];
        PC::unpack(gs[i * G + cg], u);
        PC::unpack(dzs[i * G + cg], zz);
#pragma unroll
        for (int e = 0; e < CPT; ++e) db[e] = zz[e] * sigmoid_fast(u[e]);
        dybs[i * G + cg] = fpack(db);
      }
    }
    __syncthreads();
    if (!act) continue;
    const int64_t cn = c + gridDim.x;
    if (cn < nch) {
      wins(cn, wv);
      win_load<T, CPT, U, 4>(r, src, wv, cn / nct, L, D, rr, cg, RP);
    }
    for (int i = rr; i < n; i += RP) {
      const int64_t o = (b * L + t0 + i) * D + c0;
      float zz[CPT], sg[CPT], db[CPT], ybar[CPT], dyh[CPT];
      PC::unpack(dzs[i * G + cg], zz);
      PC::unpack(gs[i * G + cg], sg);
      funpack(dybs[i * G + cg], db);
#pragma unroll
      for (int e = 0; e < CPT; ++e) sg[e] = sigmoid_fast(sg[e]);
#pragma unroll
      for (int e = 0; e < CPT; ++e) ybar[e] = dyh[e] = 0.f;
#pragma unroll
      for (int h = 0; h < HM; ++h) {
        if (h < H) {
          float yh[CPT], dp[CPT];
          PC::unpack(ys[i * G + (h * dh + j0) / CPT], yh);
          funpack(dybs[i * G + (h * dh + j0) / CPT], dp);
          const float cgh = sC[g * H + h], chg = sC[h * H + g];
          float a = 0.f;
#pragma unroll
          for (int e = 0; e < CPT; ++e) {
            ybar[e] = fmaf(cgh, yh[e], ybar[e]);
            dyh[e] = fmaf(chg, dp[e], dyh[e]);
            a = fmaf(db[e], yh[e], a);
          }
          dc[h] += a;
        }
      }
#pragma unroll
      for (int e = 0; e < CPT; ++e) ybar[e] = zz[e] * ybar[e] * sg[e] * (1.f - sg[e]);
      *reinterpret_cast<P*>(dy + o) = PC::pack(dyh);
      *reinterpret_cast<P*>(dgate + o) = PC::pack(ybar);
      if (K > 0) {
        float l[CPT], dvv[CPT];
#pragma unroll
        for (int e = 0; e < CPT; ++e) l[e] = dvv[e] = 0.f;
#pragma unroll
        for (int k = 0; k < KM; ++k)
          if (k < K) {
            float vv[CPT], za[CPT];
            PC::unpack(vs[(i + KH - k) * G + cg], vv);
            PC::unpack(dzs[(i + k) * G + cg], za);  // zero past t = L - 1
#pragma unroll
            for (int e = 0; e < CPT; ++e) {
              l[e] = fmaf(wk[k][e], vv[e], l[e]);
              dw[k][e] = fmaf(zz[e] * sc[e], vv[e], dw[k][e]);
              dvv[e] = fmaf(wk[k][e] * sc[e], za[e], dvv[e]);
            }
          }
#pragma unroll
        for (int e = 0; e < CPT; ++e) ds[e] = fmaf(zz[e], l[e], ds[e]);
        *reinterpret_cast<P*>(dv + o) = PC::pack(dvv);
      }
    }
  }
  // block partial [H*H dC | D ds | D*K dw]; sums over threads in a fixed order
  // stored column-major: entry e of this block at part[e * gridDim.x + blockIdx.x]
  auto out = [&](int e) -> float& { return part[(size_t)e * gridDim.x + blockIdx.x]; };
  float* sx = reinterpret_cast<float*>(smem);
  __syncthreads();
#pragma unroll
  for (int h = 0; h < HM; ++h)
    if (h < H) sx[threadIdx.x * H + h] = act ? dc[h] : 0.f;
  __syncthreads();
  const int gpp = dh / CPT;  // pieces per head
  for (int e = threadIdx.x; e < H * H; e += blockDim.x) {
    const int gg = e / H, h = e % H;
    float acc = 0.f;
    for (int r = 0; r < RP; ++r)
      for (int q = gg * gpp; q < (gg + 1) * gpp; ++q) acc += sx[(r * G + q) * H + h];
    out(e) = acc;
  }
  if (K == 0) return;
  __syncthreads();
  const int NX = (1 + K) * CPT;  // per thread: ds[CPT], then dw[k][CPT]
  if (act) {
#pragma unroll
    for (int e = 0; e < CPT; ++e) {
      sx[threadIdx.x * NX + e] = ds[e];
#pragma unroll
      for (int k = 0; k < KM; ++k)
        if (k < K) sx[threadIdx.x * NX + (1 + k) * CPT + e] = dw[k][e];
    }
  }
  __syncthreads();
  for (int x = threadIdx.x; x < D * (1 + K); x += blockDim.x) {
    const int c = x % D, f = x / D;  // f = 0: ds; f = 1 + k: dw[., k]
    const int q = c / CPT, e = c % CPT;
    float acc = 0.f;
    for (int r = 0; r < RP; ++r) acc += sx[(r * G + q) * NX + f * CPT + e];
    if (f == 0)
      out(H * H + c) = acc;
    else
      out(H * H + D + c * K + (f - 1)) = acc;
  }
}

// LDS bytes of the tile kernels for chunks of R rows
inline size_t epi_tile_lds(bool bwd, int D, int H, int K, int cpt, size_t es, int R) {
  const size_t KH = K > 0 ? K - 1 : 0, halo = K > 0 ? R + KH : 0;
  const size_t prm = (size_t)D * (K + 1) * 4;  // local-path parameters, before the chunk loop
  if (!bwd) {
    const size_t stage = (R + halo) * D * 4 + (size_t)R * D * es;
    return stage > prm ? stage : prm;
  }
  const size_t stage = (size_t)R * D * 4 + (2 * R + (R + KH) + halo) * D * es;
  size_t xchg = (size_t)256 * (H > (1 + K) * cpt ? H : (1 + K) * cpt) * 4;
  xchg = xchg > prm ? xchg : prm;
  return stage > xchg ? stage : xchg;
}
// Rows per chunk: each thread moves window rows rr + u RP, u < U, so a chunk and
// its K-1 halo rows fit in U RP rows; within a third of the compute unit's LDS
// (three blocks resident); 0 when no chunk fits.
constexpr size_t EPI_TILE_LDS_MAX = 53 * 1024;
inline int epi_tile_rows(bool bwd, int D, int H, int K, int cpt, size_t es) {
  const TileGeo tg = tile_geo(D, cpt);
  const int U = cpt == 1 ? tile_u<1>(bwd) : tile_u<2>(bwd);
  for (int R = U * tg.RP - (K > 0 ? K - 1 : 0); R >= 1; --R)
    if (epi_tile_lds(bwd, D, H, K, cpt, es, R) <= EPI_TILE_LDS_MAX) return R;
  return 0;
}
// channels per piece of the tile kernels for these shapes, 0 when they do not apply
template <typename T> inline int epi_tile_cpt(int vec, int D, int H, int K, bool bwd) {
  const int wide = tile_wide<T>(bwd);
  int cpt = 0;
  if (vec >= wide && K <= tile_kmax(wide) && D / wide <= 256) cpt = wide;
  else if (D <= 256) cpt = 1;
  if (cpt && epi_tile_rows(bwd, D, H, K, cpt, sizeof(T)) == 0) cpt = 0;
  return cpt;
}

// ---------------------------------------------------------------------------
static unsigned epi_grid(int64_t items) {
  const int64_t g = (items + 255) / 256;
  return (unsigned)(g < 8192 ? (g > 0 ? g : 1) : 8192);
}

template <typename T, int CPT, int HM>
static void tile_bwd(const void* y, const void* gate, const void* v, const void* dz, void* dy, void* dgate, void* dv,
                     int64_t B, int64_t L, int H, int dh, int K, const float* Ct, float lambda_c, const float* w,
                     const float* s, float* part, unsigned nparts, hipStream_t st) {
  const int R = epi_tile_rows(true, H * dh, H, K, CPT, sizeof(T));
  hipLaunchKernelGGL((epi_bwd_tile_kernel<T, CPT, HM>), dim3(nparts), dim3(256),
                     epi_tile_lds(true, H * dh, H, K, CPT, sizeof(T), R), st, (const T*)y, (const T*)gate,
                     (const T*)v, (const T*)dz, (T*)dy, (T*)dgate, (T*)dv, B, L, H, dh, K, R, Ct, lambda_c, w, s,
                     part);
}

template <typename T, int CPT, int HM, bool WL>
static void col_fwd(const void* y, const void* gate, const void* v, void* z, int64_t B, int64_t L, int H, int dh,
                    int K, const float* Ct, float lambda_c, const float* w, const float* s, hipStream_t st) {
  const int64_t np = dh / CPT, PB = np < 256 ? np : 256, RB = 256 / PB;
  const int64_t items = (B * L + RB - 1) / RB * ((np + PB - 1) / PB) * 256;  // 256 threads per block step
  const size_t lds = WL ? (size_t)H * dh * (K + 1) * sizeof(float) : 0;
  hipLaunchKernelGGL((epi_fwd_col_kernel<T, CPT, HM, WL>), dim3(epi_grid(items)), dim3(256), lds, st,
                     (const T*)y, (const T*)gate, (const T*)v, (T*)z, B * L, L, H, dh, K, Ct, lambda_c, w, s);
}

template <typename T>
hipError_t launch_epi_fwd(const void* y, const void* gate, const void* v, void* z, int64_t B, int64_t L, int H,
                          int dh, int K, const float* Ct, float lambda_c, const float* w, const float* s, int vec,
                          hipStream_t st) {
  constexpr int WIDE = 8 / sizeof(T);  // 8-byte pieces: H*CPT accumulators stay in registers
  if ((size_t)H * dh * (K + 1) * sizeof(float) > 64 * 1024)  // taps read from global memory (cached)
    col_fwd<T, 1, EPI_H_MAX, false>(y, gate, v, z, B, L, H, dh, K, Ct, lambda_c, w, s, st);
  else if (H <= 8 && vec >= WIDE && K <= 4)
    col_fwd<T, WIDE, 8, true>(y, gate, v, z, B, L, H, dh, K, Ct, lambda_c, w, s, st);
  else if (H <= 8)
    col_fwd<T, 1, 8, true>(y, gate, v, z, B, L, H, dh, K, Ct, lambda_c, w, s, st);
  else
    col_fwd<T, 1, EPI_H_MAX, true>(y, gate, v, z, B, L, H, dh, K, Ct, lambda_c, w, s, st);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_epi_bwd(const void* y, const void* gate, const void* v, const void* dz, void* dy, void* dgate,
                          void* dv, int64_t B, int64_t L, int H, int dh, int K, const float* Ct, float lambda_c,
                          const float* w, const float* s, float* dCt, float* dlambda_c, float* dw, float* ds,
                          float* part, int vec, hipStream_t st) {
  constexpr int WIDE = tile_wide<T>(true);
  const int64_t nblk = B * ((L + EPI_ROWS - 1) / EPI_ROWS);  // partial rows the workspace holds
  int64_t nparts = nblk;
  hipError_t e;
  const int cpt = epi_tile_cpt<T>(vec, H * dh, H, K, true);
  if (cpt) {
    // one partial row per block; blocks loop over chunks, so fewer blocks than chunks
    nparts = nblk < 1024 ? nblk : 1024;
    const unsigned np = (unsigned)nparts;
    if (cpt == WIDE && H <= 8)
      tile_bwd<T, WIDE, 8>(y, gate, v, dz, dy, dgate, dv, B, L, H, dh, K, Ct, lambda_c, w, s, part, np, st);
    else if (cpt == WIDE)
      tile_bwd<T, WIDE, EPI_H_MAX>(y, gate, v, dz, dy, dgate, dv, B, L, H, dh, K, Ct, lambda_c, w, s, part, np, st);
    else if (H <= 8)
      tile_bwd<T, 1, 8>(y, gate, v, dz, dy, dgate, dv, B, L, H, dh, K, Ct, lambda_c, w, s, part, np, st);
    else
      tile_bwd<T, 1, EPI_H_MAX>(y, gate, v, dz, dy, dgate, dv, B, L, H, dh, K, Ct, lambda_c, w, s, part, np, st);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  } else {
    const int64_t rows = B * L;
    const int ov = vec >= 2 ? 2 : 1;
    const int64_t items = rows * (int64_t)(H * dh / ov);
    if (ov == 2)
      hipLaunchKernelGGL((epi_bwd_act_kernel<T, 2>), dim3(epi_grid(items)), dim3(256), 0, st, (const T*)y,
                         (const T*)gate, (const T*)dz, (T*)dy, (T*)dgate, (T*)dv, rows, L, H, dh, K, Ct, lambda_c,
                         w, s);
    else
      hipLaunchKernelGGL((epi_bwd_act_kernel<T, 1>), dim3(epi_grid(items)), dim3(256), 0, st, (const T*)y,
                         (const T*)gate, (const T*)dz, (T*)dy, (T*)dgate, (T*)dv, rows, L, H, dh, K, Ct, lambda_c,
                         w, s);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL((epi_bwd_param_kernel<T>), dim3((unsigned)nblk), dim3(256), 0, st, (const T*)y,
                       (const T*)gate, (const T*)v, (const T*)dz, L, H, dh, K, w, s, part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const int P = H * H + H * dh + H * dh * K;
  double* lam_terms = reinterpret_cast<double*>(part + epi_part_floats(B, L, H, dh, K));
  hipLaunchKernelGGL(epi_bwd_reduce_kernel, dim3((unsigned)((P + 3) / 4)), dim3(256), 0, st, part, nparts, H,
                     H * dh, K, Ct, lambda_c, dCt, dw, ds, lam_terms);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(epi_bwd_lambda_kernel, dim3(1), dim3(64), 0, st, lam_terms, H, dlambda_c);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Epilogue fused with the grouped output projection (Sec. 3.4), one group per
// head and a head as wide as one MFMA contraction (32 bf16 or 16 float32
// channels):
//   out[t, g dq + o] = sum_j z[t, g dh + j] Wo[g][j][o],   z as above.
// The projection kernel's lane (token j, piece q) holds channels q VE .. q VE +
// VE-1 of a head as its activation operand; here that lane loads y, the gate and
// v at those channels of every head of its token (each element once), forms z
// of every head in registers with the arithmetic and order of the HM = 8 path of
// epi_fwd_col_kernel, rounds it as that kernel stores it, and feeds each head's
// z straight into the head's projection (gp_mma, gp_store): z never goes to
// memory, and the result is bitwise that of the epilogue followed by the
// projection.  The local path's rows t-1 and t-2 are those of lanes j-1 and j-2
// of the same 16-lane row (DPP row shifts); each lane also loads row t-3, which
// is tap 3 and, shifted left, gives the first lanes of the tile their rows
// before it.  A tap that is not in the batch row multiplies a zero weight by the
// lane's own row, as in the unfused kernel.  A wave's next tile's y rows are
// loaded before the current tile is computed and each head's gate where it is
// used, which keeps the kernel at two waves per SIMD with loads in flight while
// it computes (80 us at B4 L32K bf16 against 87 us without the prefetch).
template <typename T, int MOB, bool HASK, bool PROJ = true>
__global__ __launch_bounds__(256) void epi_proj_kernel(const T* __restrict__ y, const T* __restrict__ gate,
                                                       const T* __restrict__ v, const T* __restrict__ Wo,
                                                       T* __restrict__ out, T* __restrict__ zout, int64_t rows,
                                                       int64_t L, int H, int K,
                                                       int dq, const float* __restrict__ Ct, float lambda_c,
                                                       const float* __restrict__ w, const float* __restrict__ s) {
  typedef GPGeo<T> GG;
  constexpr int VE = GG::VE, dh = GG::KC;
  typedef Pc<T, VE> PC;
  typedef typename PC::raw P;
  extern __shared__ __align__(16) char lds[];
  const int D = H * dh, OB = dq / 16, d_out = H * dq;
  // without PROJ the kernel only writes z (the epilogue forward alone)
  char* wfrag = lds;                                                           // H * OB fragments
  float* sC = reinterpret_cast<float*>(lds + (PROJ ? (size_t)H * OB * GP_FRAG : 0));  // C [H][H]
  float* sW = sC + 64;                                                         // w as [K][D], then s [D]
  if (PROJ) gp_stage<T>(wfrag, Wo, H, dh, dq, threadIdx.x, 256);
  coupling_to_lds(sC, Ct, lambda_c, H);
  if (HASK) {
    for (int x = threadIdx.x; x < D * K; x += 256) sW[(x % K) * D + x / K] = w[x];
    for (int x = threadIdx.x; x < D; x += 256) sW[D * K + x] = s[x];
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, jj = lane & 15, q = lane >> 4, j0 = q * VE;
  const int64_t ntile = (rows + 15) / 16;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  P yr[8], yn[8];
  {
    const int64_t t = ((int64_t)blockIdx.x * 4 + wave) * 16 + jj;
    const int64_t tc = t < rows ? t : rows - 1;
#pragma unroll
    for (int h = 0; h < 8; ++h) yn[h] = *reinterpret_cast<const P*>(y + tc * D + (int64_t)(h < H ? h : 0) * dh + j0);
  }
  for (int64_t tile = (int64_t)blockIdx.x * 4 + wave; tile < ntile; tile += (int64_t)gridDim.x * 4) {
    const int64_t t = tile * 16 + jj;
    const bool tv = t < rows;
    const int64_t tc = tv ? t : rows - 1;                                   // the row loaded (any row if past the end)
    const int64_t th = t - 3 < 0 ? 0 : (t - 3 < rows ? t - 3 : rows - 1);  // row t-3 (lanes past the end included)
    const int tl = (int)(tc % L);                                           // position in the batch row
    P vm[8], vh[8];
#pragma unroll
    for (int h = 0; h < 8; ++h) yr[h] = yn[h];
    {
      const int64_t tn = t + (int64_t)gridDim.x * 64;
      const int64_t tcn = tn < rows ? tn : rows - 1;
#pragma unroll
      for (int h = 0; h < 8; ++h) yn[h] = *reinterpret_cast<const P*>(y + tcn * D + (int64_t)(h < H ? h : 0) * dh + j0);
    }
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const int hh = h < H ? h : 0;
      const int64_t c = (int64_t)hh * dh + j0;
      if (HASK) {
        vm[h] = *reinterpret_cast<const P*>(v + tc * D + c);
        vh[h] = *reinterpret_cast<const P*>(v + th * D + c);
      }
    }
#pragma unroll
    for (int g = 0; g < 8; ++g) {
      if (g >= H) continue;
      float acc[VE];
#pragma unroll
      for (int e = 0; e < VE; ++e) acc[e] = 0.f;
#pragma unroll
      for (int h = 0; h < 8; ++h) {
        float yh[VE];
        PC::unpack(yr[h], yh);
        const float cgh = h < H ? sC[g * H + h] : 0.f;
#pragma unroll
        for (int e = 0; e < VE; ++e) acc[e] = fmaf(cgh, yh[e], acc[e]);
      }
      float u[VE], o[VE];
      PC::unpack(*reinterpret_cast<const P*>(gate + tc * D + (int64_t)g * dh + j0), u);
#pragma unroll
      for (int e = 0; e < VE; ++e) o[e] = sigmoid_fast(u[e]) * acc[e];
      if (HASK) {
        const int c0 = g * dh + j0;
        float l[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) l[e] = 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const bool tap = k < K && k <= tl;
          P vk;
#pragma unroll
          for (int i = 0; i < (int)(sizeof(P) / 4); ++i) {
            uint32_t val;
            if (k == 0) {
              val = vm[g][i];
            } else if (k == 3) {
              val = vh[g][i];
            } else if (k == 1) {
              // lanes j >= k: lane j-k's own row; lanes j < k: lane j+3-k's row t-3
              // (row_shl:2 of the t-3 rows, then row_shr:1 of the own rows over it)
              const int hal = __builtin_amdgcn_update_dpp(0, (int)vh[g][i], 0x102, 0xF, 0xF, false);
              val = (uint32_t)__builtin_amdgcn_update_dpp(hal, (int)vm[g][i], 0x111, 0xF, 0xF, false);
            } else {
              const int hal = __builtin_amdgcn_update_dpp(0, (int)vh[g][i], 0x101, 0xF, 0xF, false);
              val = (uint32_t)__builtin_amdgcn_update_dpp(hal, (int)vm[g][i], 0x112, 0xF, 0xF, false);
            }
            vk[i] = tap ? val : vm[g][i];
          }
          float vv[VE];
          PC::unpack(vk, vv);
#pragma unroll
          for (int e = 0; e < VE; ++e) l[e] = fmaf(tap ? sW[k * D + c0 + e] : 0.f, vv[e], l[e]);
        }
#pragma unroll
        for (int e = 0; e < VE; ++e) o[e] = fmaf(sW[D * K + c0 + e], l[e], o[e]);
      }
      const P zp = PC::pack(o);
      if (zout != nullptr && tv) *reinterpret_cast<P*>(zout + t * D + g * dh + j0) = zp;  // z kept for a backward
      if (PROJ) {
        const u32x4 zb = __builtin_bit_cast(u32x4, zp);
        f4 a[MOB];
        const char* fb = wfrag + (size_t)g * OB * GP_FRAG + lane * 16;
#pragma unroll
        for (int ob = 0; ob < MOB; ++ob)
          if (ob < OB) a[ob] = gp_mma(*reinterpret_cast<const u32x4*>(fb + ob * GP_FRAG), zb, zero, T());
        if (tv) gp_store<T, MOB>(out + t * d_out + g * dq, a, OB, q);
      }
    }
  }
}

// bytes of LDS of the fused kernel, 0 when the shape is not one it takes
size_t epi_proj_lds(int H, int dh, int K, int64_t d_out, bool bf16) {
  const int kc = bf16 ? 32 : 16;
  if (H < 1 || H > 8 || dh != kc || K < 0 || K > 4 || d_out % H) return 0;
  const int64_t dq = d_out / H;
  if (dq != 16 && dq != 32) return 0;  // one or two output blocks per head (registers)
  const size_t lds = (size_t)H * (dq / 16) * GP_FRAG + 64 * 4 + (size_t)H * dh * (K + 1) * 4;
  return lds <= (size_t)GP_MAXLDS ? lds : 0;
}

template <typename T>
hipError_t launch_epi_proj_fwd(const void* y, const void* gate, const void* v, const void* Wo, void* out, void* z,
                               int64_t B, int64_t L, int H, int K, int64_t d_out, const float* Ct, float lambda_c,
                               const float* w, const float* s, int num_cus, hipStream_t st) {
  const size_t lds = epi_proj_lds(H, GPGeo<T>::KC, K, d_out, GPGeo<T>::BF);
  const int64_t rows = B * L, ntile = (rows + 15) / 16, want = (ntile + 3) / 4;
  const int64_t cap = (int64_t)EP_WG_PER_CU * (num_cus > 0 ? num_cus : 256);
  const dim3 grid((unsigned)(want < cap ? want : cap)), block(256);
  const int dq = (int)(d_out / H);
  if (K > 0)
    hipLaunchKernelGGL((epi_proj_kernel<T, 2, true>), grid, block, lds, st, (const T*)y, (const T*)gate, (const T*)v,
                       (const T*)Wo, (T*)out, (T*)z, rows, L, H, K, dq, Ct, lambda_c, w, s);
  else
    hipLaunchKernelGGL((epi_proj_kernel<T, 2, false>), grid, block, lds, st, (const T*)y, (const T*)gate,
                       (const T*)v, (const T*)Wo, (T*)out, (T*)z, rows, L, H, K, dq, Ct, lambda_c, w, s);
  return hipGetLastError();
}
template hipError_t launch_epi_proj_fwd<float>(const void*, const void*, const void*, const void*, void*, void*, int64_t,
                                               int64_t, int, int, int64_t, const float*, float, const float*,
                                               const float*, int, hipStream_t);
template hipError_t launch_epi_proj_fwd<bf16_t>(const void*, const void*, const void*, const void*, void*, void*, int64_t,
                                                int64_t, int, int, int64_t, const float*, float, const float*,
                                                const float*, int, hipStream_t);

// The epilogue forward alone on the fused kernel's layout (a lane holds one
// token's channels at one offset of every head, so the head mixing needs no
// exchange and the local path's earlier rows come by DPP): for H <= 8, dh = 32
// (bf16) or 16 (f32), K <= 4; z bitwise that of epi_fwd_col_kernel.
size_t epi_z_lds(int H, int dh, int K, bool bf16) {
  const int kc = bf16 ? 32 : 16;
  if (H < 1 || H > 8 || dh != kc || K < 0 || K > 4) return 0;
  return 64 * 4 + (size_t)H * dh * (K + 1) * 4;
}

template <typename T>
hipError_t launch_epi_z_fwd(const void* y, const void* gate, const void* v, void* z, int64_t B, int64_t L, int H,
                            int K, const float* Ct, float lambda_c, const float* w, const float* s, int num_cus,
                            hipStream_t st) {
  const size_t lds = epi_z_lds(H, GPGeo<T>::KC, K, GPGeo<T>::BF);
  const int64_t rows = B * L, ntile = (rows + 15) / 16, want = (ntile + 3) / 4;
  const int64_t cap = (int64_t)EP_WG_PER_CU * (num_cus > 0 ? num_cus : 256);
  const dim3 grid((unsigned)(want < cap ? want : cap)), block(256);
  if (K > 0)
    hipLaunchKernelGGL((epi_proj_kernel<T, 2, true, false>), grid, block, lds, st, (const T*)y, (const T*)gate,
                       (const T*)v, (const T*)nullptr, (T*)nullptr, (T*)z, rows, L, H, K, 16, Ct, lambda_c, w, s);
  else
    hipLaunchKernelGGL((epi_proj_kernel<T, 2, false, false>), grid, block, lds, st, (const T*)y, (const T*)gate,
                       (const T*)v, (const T*)nullptr, (T*)nullptr, (T*)z, rows, L, H, K, 16, Ct, lambda_c, w, s);
  return hipGetLastError();
}
template hipError_t launch_epi_z_fwd<float>(const void*, const void*, const void*, void*, int64_t, int64_t, int, int,
                                            const float*, float, const float*, const float*, int, hipStream_t);
template hipError_t launch_epi_z_fwd<bf16_t>(const void*, const void*, const void*, void*, int64_t, int64_t, int, int,
                                             const float*, float, const float*, const float*, int, hipStream_t);

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
