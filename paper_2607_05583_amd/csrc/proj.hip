// Grouped linear projections on MFMA (Sec. 3.1 drive and gate projection,
// Sec. 3.4 output projection): y[:, g-th output slice] = x[:, g-th input slice]
// W[g] for G groups of a block-diagonal weight W [G][d_in/G][d_out/G].
//
// There are d_in/G multiply-adds per output, so the kernel streams: a wave takes
// 16 tokens (rows of x) at a time, loads each lane's 16-byte pieces of the rows
// straight into MFMA activation operands (no LDS), and writes y from the
// accumulators.  The weights of every group are staged once per work-group in
// LDS, already in the operand layout, and read as one 16-byte fragment per lane
// and product.  With two weights (the drive and the gate of the same input) one
// read of x feeds both outputs.
//   bf16:  v_mfma_f32_16x16x32_bf16 per (group, 32 inputs, 16 outputs):
//          D = W^T x^T, lane (j, q) of the B operand holds x[t0 + j][32 kb + 8q
//          .. +7] of the group, lane (i, q) of the A operand W[32 kb + 8q + r][o(i)],
//          r = 0..7.
//   float: four v_mfma_f32_16x16x4_f32 per (group, 16 inputs, 16 outputs); the
//          r-th takes input 16 kc + 4q + r from lane (j, q)'s 16-byte piece, and
//          the A operand the matching weight rows (full float32 products).
// D lane (j, q) holds outputs o(4q + r) of token t0 + j.  Output blocks of 16 go
// in pairs, and inside a pair's 32 outputs o(i) = 8 (i / 4) + 4 (block & 1) +
// (i & 3), so that each lane ends with 8 adjacent outputs of one token (one
// 16-byte bf16 store, two float32 stores); an unpaired last block (d_out/G = 16
// mod 32) keeps o(i) = i.  float32 accumulation; bf16 outputs rounded to nearest
// even once.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "proj.h"

namespace res {

// NO weights sharing x; MP >= pieces per lane and tile, MOB >= output blocks per group
template <typename T, int NO, int MP, int MOB>
__global__ __launch_bounds__(GP_THREADS) void gproj_kernel(const T* __restrict__ x, const T* __restrict__ W0,
                                                           const T* __restrict__ W1, T* __restrict__ y0,
                                                           T* __restrict__ y1, int64_t N, int d_in, int d_out,
                                                           int G) {
  typedef GPGeo<T> GG;
  extern __shared__ __align__(16) char wfrag[];
  const int di = d_in / G, dq = d_out / G, KB = di / GG::KC, OB = dq / 16;
  const int nfrag = G * KB * OB;  // fragments of one weight
  // ---- the weights into LDS, in the operand layout ----
#pragma unroll
  for (int w = 0; w < NO; ++w)
    gp_stage<T>(wfrag + (size_t)w * nfrag * GP_FRAG, w ? W1 : W0, G, di, dq, threadIdx.x, GP_THREADS);
  __syncthreads();

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, j = lane & 15, q = lane >> 4;
  const int np = d_in / (GG::KC);  // pieces per lane and tile (one per group and fragment row)
  const int64_t ntile = (N + 15) / 16;
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  for (int64_t tile = (int64_t)blockIdx.x * 4 + wave; tile < ntile; tile += (int64_t)gridDim.x * 4) {
    const int64_t t = tile * 16 + j;
    const bool tv = t < N;
    const T* xr = x + (tv ? t : 0) * (int64_t)d_in + q * (GG::KC / 4);
    u32x4 xv[MP];
#pragma unroll
    for (int p = 0; p < MP; ++p)
      if (p < np) xv[p] = tv ? *reinterpret_cast<const u32x4*>(xr + p * GG::KC) : zero4;
    f4 acc[NO][MOB];
    int g = 0, kb = 0;
#pragma unroll
    for (int p = 0; p < MP; ++p) {
      if (p < np) {
        if (kb == 0) {
#pragma unroll
          for (int w = 0; w < NO; ++w)
#pragma unroll
            for (int ob = 0; ob < MOB; ++ob) acc[w][ob] = zero;
        }
#pragma unroll
        for (int w = 0; w < NO; ++w) {
          const char* fb = wfrag + ((size_t)w * nfrag + (size_t)p * OB) * GP_FRAG + lane * 16;
#pragma unroll
          for (int ob = 0; ob < MOB; ++ob)
            if (ob < OB)
              acc[w][ob] = gp_mma(*reinterpret_cast<const u32x4*>(fb + ob * GP_FRAG), xv[p], acc[w][ob], T());
        }
        if (kb == KB - 1 && tv) {
#pragma unroll
          for (int w = 0; w < NO; ++w) gp_store<T, MOB>((w ? y1 : y0) + t * (int64_t)d_out + g * dq, acc[w], OB, q);
        }
        if (++kb == KB) {
          kb = 0;
          ++g;
        }
      }
    }
  }
}

// Data gradient of up to three grouped projections into one input:
//   dx[t, g di + k] (+)= sum_i sum_o dy_i[t, g dq + o] W_i[g][k][o]
// (Sec. 3.1: the block input feeds the drive and the gate projections, so its
// gradient sums their data gradients).  The same streaming scheme as
// gproj_kernel with the roles of d_in and d_out exchanged: the B operand is the
// lane's 16-byte pieces of the dy_i rows, the A operand each W_i transposed in
// LDS (gp_stage_t); every input accumulates into the same accumulators, group
// by group, and the sum is rounded once (after adding dx's present value when
// ACC).
struct DgradArgs {
  const void* dy[3];
  const void* W[3];
  void* dx;
  int64_t N;
  int d_in, d_out, G;
};

template <typename T, int NI, int MP, int MOB, bool ACC>
__global__ __launch_bounds__(GP_THREADS) void gproj_dgrad_kernel(DgradArgs a) {
  typedef GPGeo<T> GG;
  extern __shared__ __align__(16) char wfrag[];
  const int di = a.d_in / a.G, dq = a.d_out / a.G, KB = dq / GG::KC, OB = di / 16;
  const int nfrag = a.G * KB * OB;  // fragments of one weight
#pragma unroll
  for (int w = 0; w < NI; ++w)
    gp_stage_t<T>(wfrag + (size_t)w * nfrag * GP_FRAG, static_cast<const T*>(a.W[w]), a.G, di, dq, threadIdx.x,
                  GP_THREADS);
  __syncthreads();

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, j = lane & 15, q = lane >> 4;
  const int np = a.d_out / GG::KC;  // pieces per lane, input and tile
  const int64_t ntile = (a.N + 15) / 16;
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  T* dx = static_cast<T*>(a.dx);
  for (int64_t tile = (int64_t)blockIdx.x * 4 + wave; tile < ntile; tile += (int64_t)gridDim.x * 4) {
    const int64_t t = tile * 16 + j;
    const bool tv = t < a.N;
    u32x4 xv[NI][MP];
#pragma unroll
    for (int w = 0; w < NI; ++w) {
      const T* xr = static_cast<const T*>(a.dy[w]) + (tv ? t : 0) * (int64_t)a.d_out + q * (GG::KC / 4);
#pragma unroll
      for (int p = 0; p < MP; ++p)
        if (p < np) xv[w][p] = tv ? *reinterpret_cast<const u32x4*>(xr + p * GG::KC) : zero4;
    }
    f4 acc[MOB];
    int g = 0, kb = 0;
#pragma unroll
    for (int p = 0; p < MP; ++p) {
      if (p < np) {
        if (kb == 0) {
#pragma unroll
          for (int ob = 0; ob < MOB; ++ob) acc[ob] = zero;
        }
#pragma unroll
        for (int w = 0; w < NI; ++w) {
          const char* fb = wfrag + ((size_t)w * nfrag + (size_t)p * OB) * GP_FRAG + lane * 16;
#pragma unroll
          for (int ob = 0; ob < MOB; ++ob)
            if (ob < OB) acc[ob] = gp_mma(*reinterpret_cast<const u32x4*>(fb + ob * GP_FRAG), xv[w][p], acc[ob], T());
        }
        if (kb == KB - 1 && tv) gp_store<T, MOB, ACC>(dx + t * (int64_t)a.d_in + g * di, acc, OB, q);
        if (++kb == KB) {
          kb = 0;
          ++g;
        }
      }
    }
  }
}

// Whether the data-gradient kernel takes n inputs of this shape: d_out/G a
// multiple of 32 (bf16) or 16 (float), d_in/G a multiple of 16 and at most 128,
// a row of dy at most 256 elements for several inputs (512 bytes for one), the
// n transposed weights at most 64 KB, and every array 16-byte aligned.
bool grouped_dgrad_supported(int n, const void* const* dy, const void* const* W, const void* dx, int64_t d_in,
                             int64_t d_out, int64_t G, bool bf16) {
  const int64_t kc = bf16 ? 32 : 16;
  const int64_t di = d_in / G, dq = d_out / G;
  if (n < 1 || n > 3 || dq % kc || di % 16 || di > 16 * GP_MAXOB) return false;
  const int64_t np = d_out / kc;
  if (np > (n == 1 ? GP_MAXP : GP_MAXP / 2)) return false;
  if ((int64_t)n * G * (dq / kc) * (di / 16) * GP_FRAG > GP_MAXLDS) return false;
  auto al = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  if (!al(dx)) return false;
  for (int i = 0; i < n; ++i)
    if (!al(dy[i]) || !al(W[i])) return false;
  return true;
}

hipError_t launch_grouped_dgrad(int n, const void* const* dy, const void* const* W, void* dx, int64_t N, int64_t d_in,
                                int64_t d_out, int64_t G, bool bf16, bool accumulate, int num_cus, hipStream_t st) {
  const int64_t kc = bf16 ? 32 : 16;
  const size_t lds = (size_t)n * G * (d_out / G / kc) * (d_in / G / 16) * GP_FRAG;
  const int64_t ntile = (N + 15) / 16, want = (ntile + 3) / 4,
                cap = (int64_t)(n == 1 ? GP_WG_PER_CU_ONE : GP_WG_PER_CU_TWO) * (num_cus > 0 ? num_cus : 256);
  const dim3 grid((unsigned)(want < cap ? want : cap)), block(GP_THREADS);
  DgradArgs a{};
  for (int i = 0; i < 3; ++i) {
    a.dy[i] = i < n ? dy[i] : dy[0];
    a.W[i] = i < n ? W[i] : W[0];
  }
  a.dx = dx;
  a.N = N;
  a.d_in = (int)d_in;
  a.d_out = (int)d_out;
  a.G = (int)G;
  const int np = (int)(d_out / kc), nob = (int)(d_in / G / 16);
  auto go = [&](auto tag, auto ni_, auto mp_, auto mob_, auto acc_) {
    typedef decltype(tag) T;
    constexpr int NI = decltype(ni_)::value, MP = decltype(mp_)::value, MOB = decltype(mob_)::value;
    constexpr bool ACC = decltype(acc_)::value;
    hipLaunchKernelGGL((gproj_dgrad_kernel<T, NI, MP, MOB, ACC>), grid, block, lds, st, a);
  };
  typedef std::integral_constant<int, 1> I1;
  typedef std::integral_constant<int, 2> I2;
  typedef std::integral_constant<int, 3> I3;
  typedef std::integral_constant<int, 8> I8;
  typedef std::integral_constant<int, 16> I16;
  typedef std::integral_constant<bool, true> BT;
  typedef std::integral_constant<bool, false> BFa;
  auto by_mob = [&](auto tag, auto ni_, auto mp_, auto acc_) {
    if (nob <= 2) go(tag, ni_, mp_, I2(), acc_); else go(tag, ni_, mp_, I8(), acc_);
  };
  auto by_n = [&](auto tag, auto acc_) {
    if (n == 1) {
      if (np <= 8) by_mob(tag, I1(), I8(), acc_); else by_mob(tag, I1(), I16(), acc_);
    } else if (n == 2) {
      by_mob(tag, I2(), I8(), acc_);
    } else {
      by_mob(tag, I3(), I8(), acc_);
    }
  };
  auto by_acc = [&](auto tag) {
    if (accumulate) by_n(tag, BT()); else by_n(tag, BFa());
  };
  if (bf16) by_acc(bf16_t()); else by_acc(float());
  return hipGetLastError();
}

// Weight gradient of grouped projections of one input x (bf16), summed over up
// to three output gradients into one or two weights:
//   dW_m[g][k][o] (+)= sum_t x[t, g di + k] sum_{i: out(i) = m} dy_i[t, g dq + o]
// The contraction runs over the tokens, so an MFMA operand lane needs 8
// consecutive tokens of one channel.  A work-group stages chunks of 32 tokens of
// x and of each dy_i in LDS channel-major: a thread loads an 8 x 8 block (8 rows'
// 16-byte pieces of 8 channels, prefetched into registers one chunk ahead),
// transposes it in registers and writes 8 channel pieces of 16 bytes.  Channel c
// sits at column position c ^ ((c / 8) mod 4) (64 bytes a column), which spreads
// the block writes over all banks and keeps the 16 channels of one operand read
// in one contiguous kilobyte; every operand is then one 16-byte LDS read.
// Output blocks of 16 x 16 (per weight, group, input block kb and output block
// ob) are split over the eight waves; block (k, o) of lane (j, q) holds rows
// 4q + r, column j.  Each work-group writes its token range's sums as partials;
// wgrad_reduce_kernel adds them over the work-groups in a fixed order
// (deterministic).
struct WgradArgs {
  const void* x;
  const void* dy[3];
  float* part;
  int64_t N, tpw;  // tokens, tokens per work-group (a multiple of 32)
  int d_in, d_out, G, omap, nb;  // omap bit i: the weight input i adds to; nb: output blocks
};

__device__ __forceinline__ int wt_pos(int c) { return c ^ ((c >> 3) & 3); }

template <int NI>
__global__ __launch_bounds__(WT_THREADS) void gproj_wgrad_kernel(WgradArgs a) {
  extern __shared__ __align__(16) char lds[];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, li = lane & 15, lq = lane >> 4;
  const int di = a.d_in / a.G, dq = a.d_out / a.G, KB = di / 16, OB = dq / 16, per_w = a.G * KB * OB;
  char* xs = lds;
  char* ys = lds + a.d_in * 64;  // input i at ys + i d_out 64
  const int per = (a.nb + WT_WAVES - 1) / WT_WAVES, b0 = wave * per, b1 = b0 + per < a.nb ? b0 + per : a.nb;
  const int64_t tb = (int64_t)blockIdx.x * a.tpw, te = tb + a.tpw < a.N ? tb + a.tpw : a.N;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  f4 acc[WT_MAXB];
#pragma unroll
  for (int s = 0; s < WT_MAXB; ++s) acc[s] = zero;
  // 8 x 8 blocks: x has 4 (row blocks) x d_in / 8 of them, each dy_i 4 x d_out / 8
  const int nbx = a.d_in / 2, nby = a.d_out / 2, nbt = nbx + NI * nby;
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
  u32x4 rv[WT_MAXU][8];
  auto src = [&](int e, const bf16_t*& base, int& d, int& cb, int& rb, char*& dst) {
    int t = e, k = 0;
    if (t >= nbx) {
      t -= nbx;
      k = 1 + t / nby;
      t = t % nby;
    }
    d = k ? a.d_out : a.d_in;
    base = static_cast<const bf16_t*>(k ? a.dy[k - 1 < NI ? k - 1 : 0] : a.x);
    dst = k ? ys + (k - 1) * a.d_out * 64 : xs;
    cb = t % (d / 8);
    rb = t / (d / 8);
  };
  auto load = [&](int64_t t0) {
#pragma unroll
    for (int u = 0; u < WT_MAXU; ++u) {
      const int e = tid + WT_THREADS * u;
      if (e < nbt) {
        const bf16_t* base;
        int d, cb, rb;
        char* dst;
        src(e, base, d, cb, rb, dst);
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          const int64_t t = t0 + 8 * rb + r;
          rv[u][r] = t < te ? *reinterpret_cast<const u32x4*>(base + t * d + 8 * cb) : zero4;
        }
      }
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int u = 0; u < WT_MAXU; ++u) {
      const int e = tid + WT_THREADS * u;
      if (e < nbt) {
        const bf16_t* base;
        int d, cb, rb;
        char* dst;
        src(e, base, d, cb, rb, dst);
        (void)base;
#pragma unroll
        for (int k = 0; k < 8; ++k) {  // channel 8 cb + k: rows 8 rb .. 8 rb + 7
          u32x4 o;
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            const uint32_t lo = rv[u][2 * h][k >> 1], hi = rv[u][2 * h + 1][k >> 1];
            o[h] = (k & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
          }
          *reinterpret_cast<u32x4*>(dst + wt_pos(8 * cb + k) * 64 + rb * 16) = o;
        }
      }
    }
  };
  if (tb < te) load(tb);
  for (int64_t t0 = tb; t0 < te; t0 += WT_T) {
    __syncthreads();  // the previous chunk's operand reads are done
    store();
    __syncthreads();
    if (t0 + WT_T < te) load(t0 + WT_T);
#pragma unroll
    for (int s = 0; s < WT_MAXB; ++s) {
      const int b = b0 + s;
      if (b < b1) {
        const int m = b / per_w, rem = b % per_w, g = rem / (KB * OB), kb = (rem / OB) % KB, ob = rem % OB;
        const u32x4 A = *reinterpret_cast<const u32x4*>(xs + wt_pos(g * di + kb * 16 + li) * 64 + lq * 16);
        const int cy = wt_pos(g * dq + ob * 16 + li) * 64 + lq * 16;
#pragma unroll
        for (int i = 0; i < NI; ++i)
          if (((a.omap >> i) & 1) == m)
            acc[s] = gp_mma(A, *reinterpret_cast<const u32x4*>(ys + i * a.d_out * 64 + cy), acc[s], bf16_t());
      }
    }
  }
#pragma unroll
  for (int s = 0; s < WT_MAXB; ++s) {
    const int b = b0 + s;
    if (b < b1) *reinterpret_cast<f4*>(a.part + (((size_t)blockIdx.x * a.nb + b) * 64 + lane) * 4) = acc[s];
  }
}

// dW_m entries from the partials of nwg work-groups: a block takes 32 entries,
// its eight slices of 32 threads sum every eighth work-group's partial (slice
// k: work-groups k, k + 8, ...) in order, and the slices' sums are added in
// slice order, so the result does not depend on the launch.
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float* __restrict__ P, float* __restrict__ dW0,
                                                           float* __restrict__ dW1, int nwg, int nb, int G, int di,
                                                           int dq, int accumulate) {
  __shared__ float sp[8][32];
  const int KB = di / 16, OB = dq / 16, per_w = G * KB * OB;
  const int el = threadIdx.x & 31, sl = threadIdx.x >> 5;
  const int64_t E = (int64_t)nb * 256, e = (int64_t)blockIdx.x * 32 + el;
  float v = 0.f;
  if (e < E) {
#pragma unroll 8
    for (int w = sl; w < nwg; w += 8) v += P[(size_t)w * E + e];
  }
  sp[sl][el] = v;
  __syncthreads();
  if (sl != 0 || e >= E) return;
#pragma unroll
  for (int k = 1; k < 8; ++k) v += sp[k][el];
  const int b = (int)(e >> 8), lane = (int)(e >> 2) & 63, r = (int)e & 3, j = lane & 15, q = lane >> 4;
  const int m = b / per_w, rem = b % per_w, g = rem / (KB * OB), kb = (rem / OB) % KB, ob = rem % OB;
  float* W = m ? dW1 : dW0;
  const size_t idx = ((size_t)g * di + kb * 16 + 4 * q + r) * dq + ob * 16 + j;
  W[idx] = accumulate ? W[idx] + v : v;
}

// Output blocks of the weight-gradient kernel, 0 when it does not take the shape
// (bf16; d_in and d_out multiples of 64 and at most 256; d_in/G and d_out/G
// multiples of 16; at most 64 blocks of 16 x 16; the chunk at most 64 KB of LDS).
int grouped_wgrad_blocks(int n, int nout, int64_t d_in, int64_t d_out, int64_t G, bool bf16) {
  if (!bf16 || n < 1 || n > 3 || nout < 1 || nout > 2 || G < 1 || d_in % G || d_out % G) return 0;
  const int64_t di = d_in / G, dq = d_out / G;
  if (d_in % 64 || d_out % 64 || d_in > 256 || d_out > 256 || di % 16 || dq % 16) return 0;
  const int64_t nb = nout * G * (di / 16) * (dq / 16);
  if (nb > WT_WAVES * WT_MAXB || (int64_t)WT_T * (d_in + n * d_out) * 2 > GP_MAXLDS) return 0;
  if ((d_in + n * d_out) / 2 > WT_THREADS * WT_MAXU) return 0;
  return (int)nb;
}

// Work-groups: at least WT_MIN_TOKENS tokens each; at most WT_GRID, or twice
// as many for one gradient (half the chunk bytes per work-group, so two
// work-groups per compute unit keep as many loads in flight).
int64_t grouped_wgrad_grid(int64_t N, int n) {
  const int64_t cap = n == 1 ? 2 * WT_GRID : WT_GRID;
  const int64_t g = (N + WT_MIN_TOKENS - 1) / WT_MIN_TOKENS;
  return g < 1 ? 1 : (g > cap ? cap : g);
}

hipError_t launch_grouped_wgrad(int n, const void* x, const void* const* dy, const int* out, float* dW0, float* dW1,
                                int64_t N, int64_t d_in, int64_t d_out, int64_t G, bool accumulate, float* part,
                                hipStream_t st) {
  int nout = 1, omap = 0;
  for (int i = 0; i < n; ++i) {
    omap |= (out[i] & 1) << i;
    if (out[i] == 1) nout = 2;
  }
  WgradArgs a{};
  a.x = x;
  for (int i = 0; i < 3; ++i) a.dy[i] = i < n ? dy[i] : dy[0];
  a.part = part;
  a.N = N;
  a.d_in = (int)d_in;
  a.d_out = (int)d_out;
  a.G = (int)G;
  a.omap = omap;
  a.nb = grouped_wgrad_blocks(n, nout, d_in, d_out, G, true);
  const int64_t grid = grouped_wgrad_grid(N, n);
  a.tpw = ((N + grid - 1) / grid + WT_T - 1) / WT_T * WT_T;
  const size_t lds = (size_t)WT_T * (d_in + n * d_out) * 2;
  if (n == 1)
    hipLaunchKernelGGL(gproj_wgrad_kernel<1>, dim3((unsigned)grid), dim3(WT_THREADS), lds, st, a);
  else if (n == 2)
    hipLaunchKernelGGL(gproj_wgrad_kernel<2>, dim3((unsigned)grid), dim3(WT_THREADS), lds, st, a);
  else
    hipLaunchKernelGGL(gproj_wgrad_kernel<3>, dim3((unsigned)grid), dim3(WT_THREADS), lds, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t E = (int64_t)a.nb * 256;
  hipLaunchKernelGGL(wgrad_reduce_kernel, dim3((unsigned)((E + 31) / 32)), dim3(256), 0, st, part, dW0,
                     nout == 2 ? dW1 : dW0, (int)grid, a.nb, (int)G, (int)(d_in / G), (int)(d_out / G),
                     (int)accumulate);
  return hipGetLastError();
}

// Whether the MFMA kernel takes this shape: d_in/G a multiple of 32 (bf16) or 16
// (float), d_out/G a multiple of 16 and at most 128, a row of x at most 1 KB, the
// staged weights at most 64 KB, and x and the outputs 16-byte aligned.
bool grouped_proj_supported(const void* x, const void* W0, const void* W1, const void* y0, const void* y1,
                            int64_t d_in, int64_t d_out, int64_t G, bool bf16) {
  const int nw = W1 ? 2 : 1;
  const int64_t es = bf16 ? 2 : 4, kc = bf16 ? 32 : 16;
  const int64_t di = d_in / G, dq = d_out / G;
  if (di % kc || dq % 16 || dq > 16 * GP_MAXOB || d_in * es > 16 * 4 * GP_MAXP) return false;
  if ((int64_t)nw * G * (di / kc) * (dq / 16) * GP_FRAG > GP_MAXLDS) return false;
  auto al = [](const void* p) { return p == nullptr || ((uintptr_t)p & 15) == 0; };
  return al(x) && al(W0) && al(W1) && al(y0) && al(y1);
}

hipError_t launch_grouped_proj(const void* x, const void* W0, const void* W1, void* y0, void* y1, int64_t N,
                               int64_t d_in, int64_t d_out, int64_t G, bool bf16, int num_cus, hipStream_t st) {
  const int nw = W1 ? 2 : 1;
  const int64_t kc = bf16 ? 32 : 16;
  const size_t lds = (size_t)nw * G * (d_in / G / kc) * (d_out / G / 16) * GP_FRAG;
  const int64_t ntile = (N + 15) / 16, want = (ntile + 3) / 4, cap = (int64_t)(nw == 1 ? GP_WG_PER_CU_ONE : GP_WG_PER_CU_TWO) * (num_cus > 0 ? num_cus : 256);
  const dim3 grid((unsigned)(want < cap ? want : cap)), block(GP_THREADS);
  const int di = (int)d_in, dq = (int)d_out, g = (int)G;
  const int np = (int)(d_in / kc), nob = (int)(d_out / G / 16);
  auto go = [&](auto tag, auto no_, auto mp_, auto mob_) {
    typedef decltype(tag) T;
    constexpr int NO = decltype(no_)::value, MP = decltype(mp_)::value, MOB = decltype(mob_)::value;
    const T* w0 = (const T*)W0;
    hipLaunchKernelGGL((gproj_kernel<T, NO, MP, MOB>), grid, block, lds, st, (const T*)x, w0, NO == 2 ? (const T*)W1 : w0,
                       (T*)y0, NO == 2 ? (T*)y1 : (T*)y0, N, di, dq, g);
  };
  typedef std::integral_constant<int, 1> I1;
  typedef std::integral_constant<int, 2> I2;
  typedef std::integral_constant<int, 8> I8;
  typedef std::integral_constant<int, 16> I16;
  auto by_shape = [&](auto tag, auto no_) {
    if (np <= 8) {
      if (nob <= 2) go(tag, no_, I8(), I2()); else go(tag, no_, I8(), I8());
    } else {
      if (nob <= 2) go(tag, no_, I16(), I2()); else go(tag, no_, I16(), I8());
    }
  };
  if (bf16) {
    if (nw == 2) by_shape(bf16_t(), I2()); else by_shape(bf16_t(), I1());
  } else {
    if (nw == 2) by_shape(float(), I2()); else by_shape(float(), I1());
  }
  return hipGetLastError();
}

}  // namespace res
