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
