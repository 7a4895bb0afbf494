// Forward resonant mixing, prompt state and parameter tables for gfx950.
//
// Operator (Sec. 3.1 kernel, Sec. 3.2 causal convolution, Sec. 3.3 recurrence):
//   y[t] = sum_{s<=t} K[t-s] x[s] + Re sum_m c_m lambda_m^(t+1) h0_m,
//   K[tau] = Re sum_m c_m lambda_m^tau.
// Chunked form used here (chunk of CHUNK = 16 steps, chunk n starts at 16 n):
//   y_loc[16n+i] = sum_{k<=i} K[i-k] x[16n+k]                 T  (16x16 lower Toeplitz)
//   S_m[n]      = sum_k lambda_m^(15-k) x[16n+k]              V  (16 x 16: 8 modes, re/im)
//   H_m[n+1]    = lambda_m^16 H_m[n] + S_m[n]                  scan over chunks
//   y[16n+i]    = y_loc[16n+i] + Re sum_m c_m lambda_m^(i+1) H_m[n]   U (16 x 16)
// where H_m[n] is the state entering chunk n.  Per channel the three products
// are 16x16 MFMAs whose 16 columns are the chunks of one tile (256 steps); all
// chunks share the per-channel matrices because the filter is time invariant.
// Inside a tile the chunk scan runs one lane per (channel, mode).  Across tiles
// the state is chained in a single pass (decoupled look-back): each tile
// publishes the end state of its own drives, then the state entering it,
// computed from its predecessors' published states.
#include "common.h"
#include "kernels.h"
#include "tile_io.h"

namespace res {

// ---------------------------------------------------------------------------
// Parameter tables.  One block per (padded) channel.  Every power lambda^n used
// (n = 0..16, 128, 256, last_len) is evaluated directly as
// exp(-gamma n) (cos(omega n), sin(omega n)) in float64 from the exact
// products gamma n and omega n (float32 times a small integer), and c =
// a (cos phi, sin phi); all are independent, so the block does them in
// parallel.  Entries are rounded once to the operand type.
// ---------------------------------------------------------------------------
template <typename TA, bool BWD>
__global__ __launch_bounds__(256) void prep_kernel(const float* __restrict__ gamma,
                                                   const float* __restrict__ omega,
                                                   const float* __restrict__ amp,
                                                   const float* __restrict__ phase, int D, int M,
                                                   int MG, int last_len, int seg_steps,
                                                   TA* __restrict__ tab,
                                                   ModeScalars* __restrict__ scal,
                                                   ModeCarry* __restrict__ cc,
                                                   float2* __restrict__ mpow,
                                                   float2* __restrict__ spow,
                                                   uint32_t* __restrict__ flags, int64_t nflags) {
  // lambda^0..16, then lambda^128, lambda^256, lambda^last_len
  constexpr int NPW = CHUNK + 1 + 3;
  const int d = blockIdx.x;
  const int Mp = MODES_PER_GROUP * MG;
  __shared__ double2 pw[MODES_PER_GROUP * MG_MAX][NPW];
  __shared__ double2 cm[MODES_PER_GROUP * MG_MAX];  // c
  __shared__ double taps[CHUNK + 1];

  if (flags != nullptr)  // segment flags of the single-kernel forward
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nflags;
         i += (int64_t)gridDim.x * blockDim.x)
      flags[i] = FLAG_NONE;
  const bool dvalid = d < D;
  for (int t = threadIdx.x; t < Mp * (NPW + 1); t += blockDim.x) {
    const int m = t / (NPW + 1), k = t % (NPW + 1);
    const bool valid = dvalid && m < M;
    if (k < NPW) {
      const int n = k <= CHUNK          ? k
                    : k == CHUNK + 1 ? TILE_T / 2
                    : k == CHUNK + 2 ? TILE_T
                                     : last_len;
      double2 z = make_double2(0.0, 0.0);
      if (valid) {
        double sn, cs;
        sincos((double)omega[d * M + m] * n, &sn, &cs);
        const double e = exp(-(double)gamma[d * M + m] * n);
        z = make_double2(e * cs, e * sn);
      }
      pw[m][k] = z;
    } else {
      double2 z = make_double2(0.0, 0.0);
      if (valid) {
        double sn, cs;
        sincos((double)phase[d * M + m], &sn, &cs);
        const double av = (double)amp[d * M + m];
        z = make_double2(av * cs, av * sn);
      }
      cm[m] = z;
    }
  }
  __syncthreads();
  for (int m = threadIdx.x; m < Mp; m += blockDim.x) {
    const double2 lam = pw[m][1], lH = pw[m][CHUNK + 1], lT = pw[m][CHUNK + 2];
    ModeScalars ms;
    ms.lam = make_float2((float)lam.x, (float)lam.y);
    ms.mu = make_float2((float)pw[m][CHUNK].x, (float)pw[m][CHUNK].y);
    ms.mu8 = make_float2((float)lH.x, (float)lH.y);
    ms.lamT = make_float2((float)lT.x, (float)lT.y);
    scal[(size_t)d * Mp + m] = ms;
    ModeCarry mc;
    mc.lamT = lT;
    mc.lamEll = pw[m][CHUNK + 3];
    mc.mu8 = lH;
    cc[(size_t)d * Mp + m] = mc;
  }
  if (mpow != nullptr)  // lambda^(16 j), j = 0..15, as [d][j][Mp]
    for (int t = threadIdx.x; t < CHUNK * Mp; t += blockDim.x) {
      const int j = t / Mp, m = t % Mp;
      float2 z = make_float2(0.f, 0.f);
      if (dvalid && m < M) {
        double sn, cs;
        sincos((double)omega[d * M + m] * (CHUNK * j), &sn, &cs);
        const double e = exp(-(double)gamma[d * M + m] * (CHUNK * j));
        z = make_float2((float)(e * cs), (float)(e * sn));
      }
      mpow[((size_t)d * CHUNK + j) * Mp + m] = z;
    }
  if (spow != nullptr)  // lambda^(seg_steps n), n = 0..16, as [d][n][Mp]
    for (int t = threadIdx.x; t < (CHUNK + 1) * Mp; t += blockDim.x) {
      const int n = t / Mp, m = t % Mp;
      float2 z = make_float2(0.f, 0.f);
      if (dvalid && m < M) {
        double sn, cs;
        sincos((double)omega[d * M + m] * ((double)seg_steps * n), &sn, &cs);
        const double e = exp(-(double)gamma[d * M + m] * ((double)seg_steps * n));
        z = make_float2((float)(e * cs), (float)(e * sn));
      }
      spow[((size_t)d * (CHUNK + 1) + n) * Mp + m] = z;
    }
  for (int tau = threadIdx.x; tau <= CHUNK; tau += blockDim.x) {  // K[tau] = Re sum_m c lambda^tau
    double s = 0.0;
    for (int m = 0; m < Mp; ++m) s += cm[m].x * pw[m][tau].x - cm[m].y * pw[m][tau].y;
    taps[tau] = s;
  }
  __syncthreads();

  auto part = [](double2 z, int p) { return p ? z.y : z.x; };
  // entry (mat, i, k) of the per-channel 16x16 matrices, k = contraction index
  auto entry = [&](int mat, int i, int k) -> double {
    if (!BWD) {
      if (mat == 0) return (i >= k) ? taps[i - k] : 0.0;          // T[i][k] = K[i-k]
      const int g = (mat - 1) / 2;
      if ((mat - 1) % 2 == 0)                                     // V[comp i][k] = lambda^(15-k)
        return part(pw[g * 8 + i / 2][CHUNK - 1 - k], i & 1);
      const int m = g * 8 + k / 2;                                // U[i][comp k] = c lambda^(i+1)
      const double2 z = zmul(cm[m], pw[m][i + 1]);
      return (k & 1) ? -z.y : z.x;
    }
    if (mat == 0) return (k >= i) ? taps[k - i] : 0.0;            // Tt[j=i][k] = K[k-i]
    const int g = (mat - 1) / 5, s = (mat - 1) % 5;
    const int mi = g * 8 + i / 2;
    switch (s) {
      case 0: return part(pw[mi][k], i & 1);                      // Eq[comp i][k] = lambda^k
      case 1: return k * part(pw[mi][k], i & 1);                  // Er = k lambda^k
      case 2: return part(pw[mi][CHUNK - k], i & 1);              // Xs = lambda^(16-k)
      case 3: return (CHUNK - k) * part(pw[mi][CHUNK - k], i & 1);  // Xw = (16-k) lambda^(16-k)
      default: {                                                  // Ub[j=i][comp k] = c lambda^(16-i)
        const int m = g * 8 + k / 2;
        const double2 z = zmul(cm[m], pw[m][CHUNK - i]);
        return (k & 1) ? -z.y : z.x;
      }
    }
  };

  // Store in the per-lane operand layout: 16 bytes per lane.
  const int nm = BWD ? bwd_mats(MG) : fwd_mats(MG);
  for (int task = threadIdx.x; task < nm * 64; task += blockDim.x) {
    const int mat = task / 64, l = task % 64, i = l % 16, q = l / 16;
    const bool state_mat = BWD ? bwd_mat_is_state(mat) : fwd_mat_is_state(mat);
    uint4 out;
    if (sizeof(TA) == 4 || state_mat) {
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) v[r] = (float)entry(mat, i, 4 * q + r);
      out = *reinterpret_cast<const uint4*>(v);
    } else {
      bf16_t v[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const double e = entry(mat, i, 8 * (q & 1) + r);
        const bf16_t hi = from_f32<bf16_t>((float)e);
        v[r] = (q < 2) ? hi : from_f32<bf16_t>((float)(e - (double)to_f32(hi)));
      }
      out = *reinterpret_cast<const uint4*>(v);
    }
    static_assert(sizeof(uint4) == TAB_LANE_BYTES, "one table lane is 16 bytes");
    reinterpret_cast<uint4*>(tab)[((size_t)d * nm + mat) * 64 + l] = out;
  }
}

// ---------------------------------------------------------------------------
// Forward tile machinery.
//
// A tile is one batch row b, 256 steps and DW channels (64 bf16 / 32 fp32, so a
// time row of the tile is one 128-byte segment).  Four waves each own CPW = DW/4
// channels, handled in groups of 4.
//
// LDS.  The drive tile is time-major: 32 groups of 8 rows (128 B each) with a
// 4-byte pad per group, filled by direct-to-LDS 16-byte loads.  Each output
// channel overwrites its own drive column once its products are done, and the
// tile leaves as 16-byte row stores.  Each wave has a scan buffer
// [4 channels][16 chunks][16 MG floats]: chunk states go from the MFMA layout
// (lane (n, q) holds components 4q..4q+3 of chunk n) to the scan layout, and
// the carried states come back the same way.
//
// Scan layout: lane 16 c + 2 m + h holds channel c of the group, mode m, for the
// chunk half h (chunks 8h .. 8h+7).  With A_h the end state of half h from a
// zero start (A_h = sum_j mu^(7-j) S[8h+j], mu = lambda^16), the tile's own
// end state is mu^8 A_0 + A_1, and half 1 of a tile entered with state c enters
// with mu^8 c + A_0.
//
// Per-tile records ([tile][DW * Mp] float4, slot q = wave * 32 PAIRS + 32 (grp
// MG + g) + 8 c + m): the aggregate kernel writes (A_0, A_1); the carry kernel
// writes the entry states (c, mu^8 c + A_0) of both halves.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

// Time-major LDS tile of elements of ES bytes: rows of 128 bytes (the tile's
// channels), groups of 8 rows padded so that every group starts on a 16-byte
// boundary for the direct-to-LDS loads and row stores (bf16: +8 bytes, so the
// 8-byte operand gathers of 16 lanes from 16 different groups spread over the
// banks; float: +16 bytes).
constexpr int XROW = 128;
template <int ES> struct XLay {
  static constexpr int GRP = 8 * XROW + (ES == 2 ? 8 : 16);
  static constexpr int BYTES = (TILE_T / 8) * GRP;
  __device__ static __forceinline__ int off(int t) { return (t >> 3) * GRP + (t & 7) * XROW; }
};

// Compiler-level ordering of LDS accesses inside one wave (the LDS executes a
// wave's accesses in program order).
__device__ __forceinline__ void wave_lds_order() { asm volatile("" ::: "memory"); }

// Drive tile [t0, t0 + 256) x [d0, d0 + DW) of row b into the time-major LDS
// tile; zeros outside [0, L) x [0, D).  full: the whole tile is in range and the
// rows are 16-byte aligned (direct-to-LDS loads); the caller waits (vmcnt) and
// synchronises before reading.
template <typename TX>
__device__ __forceinline__ void tile_load(char* xt, const TX* x, int64_t b, int64_t t0, int d0,
                                          int64_t L, int D, bool full, int tid) {
  constexpr int DW = tile_channels<TX>(), XE = (int)sizeof(TX);
  const int lane = tid & 63, wave = tid >> 6;
  if (full) {
    const char* src = reinterpret_cast<const char*>(x) + ((b * L + t0) * D + d0) * XE;
    const int64_t rowb = (int64_t)D * XE;
#pragma unroll
    for (int i = 0; i < TILE_T / 8 / NWAVES; ++i) {
      const int g = wave * (TILE_T / 8 / NWAVES) + i;
      const char* s = src + (int64_t)(8 * g + (lane >> 3)) * rowb + (lane & 7) * 16;
      __builtin_amdgcn_global_load_lds((gvoid_t*)s, (lvoid_t*)(xt + g * XLay<XE>::GRP), 16, 0, 0);
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += NTHREADS) {
      const int t = idx / DW, c = idx % DW;
      TX v = from_f32<TX>(0.f);
      if (t0 + t < L && d0 + c < D) v = x[(b * L + t0 + t) * (int64_t)D + d0 + c];
      *reinterpret_cast<TX*>(xt + XLay<XE>::off(t) + c * XE) = v;
    }
  }
}

template <typename TY>
__device__ __forceinline__ void tile_store(TY* y, const char* xt, int64_t b, int64_t t0, int d0,
                                           int64_t L, int D, bool full, int tid) {
  constexpr int DW = tile_channels<TY>(), YE = (int)sizeof(TY);
  const int lane = tid & 63, wave = tid >> 6;
  if (full) {
    char* dst = reinterpret_cast<char*>(y) + ((b * L + t0) * D + d0) * YE;
    const int64_t rowb = (int64_t)D * YE;
#pragma unroll
    for (int i = 0; i < TILE_T / 8 / NWAVES; ++i) {
      const int g = wave * (TILE_T / 8 / NWAVES) + i;
      const uint4 v = *reinterpret_cast<const uint4*>(xt + g * XLay<YE>::GRP + lane * 16);
      *reinterpret_cast<uint4*>(dst + (int64_t)(8 * g + (lane >> 3)) * rowb + (lane & 7) * 16) = v;
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += NTHREADS) {
      const int t = idx / DW, c = idx % DW;
      if (t0 + t < L && d0 + c < D)
        y[(b * L + t0 + t) * (int64_t)D + d0 + c] = *reinterpret_cast<const TY*>(xt + XLay<YE>::off(t) + c * YE);
    }
  }
}

// Activation operand of chunk n for channel ch from the time-major tile.
// Activations of the 4 consecutive channels ch0 .. ch0+3 (ch0 a multiple of 4)
// as MFMA B operands, one LDS read of the 4 channels per tile row.
template <typename TX> struct XGather;
template <> struct XGather<bf16_t> {
  // lane (n, q): taps 8(q&1) .. +7 = rows 16n + 8(q&1) + r = group 2n + (q&1), row r
  __device__ static __forceinline__ void get4(const char* xt, int ch0, int n, int q, bf8 (&xv)[4]) {
    const char* p = xt + (2 * n + (q & 1)) * XLay<2>::GRP + ch0 * 2;
    uint2 w[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) w[r] = *reinterpret_cast<const uint2*>(p + r * XROW);
    // channel c of row r is the (c & 1) half of word c >> 1 of w[r]
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      uint32_t o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t lo = (c >> 1) ? w[2 * j].y : w[2 * j].x;
        const uint32_t hi = (c >> 1) ? w[2 * j + 1].y : w[2 * j + 1].x;
        o[j] = (c & 1) ? ((lo >> 16) | (hi & 0xFFFF0000u)) : ((lo & 0xFFFFu) | (hi << 16));
      }
      xv[c] = __builtin_bit_cast(bf8, *reinterpret_cast<const uint4*>(o));
    }
  }
};
template <> struct XGather<float> {
  // lane (n, q), slot kk: tap 4q + kk = row 16n + 4q + kk = group 2n + (q>>1), row 4(q&1) + kk
  __device__ static __forceinline__ void get4(const char* xt, int ch0, int n, int q, f4 (&xv)[4]) {
    const char* p = xt + (2 * n + (q >> 1)) * XLay<4>::GRP + 4 * (q & 1) * XROW + ch0 * 4;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const f4 w = *reinterpret_cast<const f4*>(p + kk * XROW);
#pragma unroll
      for (int c = 0; c < 4; ++c) xv[c][kk] = w[c];
    }
  }
};

// Outputs of the 4 consecutive channels ch0 .. ch0+3 of a group (MFMA D layout,
// lane (n, q) holds rows 16n + 4q + r) into the time-major LDS tile.
template <typename TY>
__device__ __forceinline__ void put_y4(char* xt, int ch0, int n, int q, const f4 (&acc)[4]) {
  // rows 16n + 4q + r: group 2n + (q >> 1), rows 4 (q & 1) + r
  char* dst = xt + (2 * n + (q >> 1)) * XLay<sizeof(TY)>::GRP + 4 * (q & 1) * XROW + ch0 * (int)sizeof(TY);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (sizeof(TY) == 2) {
      typedef __bf16 bf4 __attribute__((ext_vector_type(4)));
      const bf4 v = {(__bf16)acc[0][r], (__bf16)acc[1][r], (__bf16)acc[2][r], (__bf16)acc[3][r]};
      *reinterpret_cast<bf4*>(dst + r * XROW) = v;
    } else {
      const f4 v = {acc[0][r], acc[1][r], acc[2][r], acc[3][r]};
      *reinterpret_cast<f4*>(dst + r * XROW) = v;
    }
  }
}

__device__ __forceinline__ float swap_pair(float v) {  // value of the neighbouring lane (lane ^ 1)
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1,
                                                               0xF, 0xF, false));
}

// float32 outputs straight from the MFMA registers: rows t .. t+3 of the 4
// channels d .. d+3, 16 bytes per row where all 4 channels exist.
__device__ __forceinline__ void put_y4_global(float* y, const f4 (&acc)[4], int64_t b, int64_t t, int d,
                                              int64_t L, int D) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (t + r >= L) break;
    float* dst = y + (b * L + t + r) * (int64_t)D + d;
    if (d + 4 <= D && (D & 3) == 0) {
      const f4 v = {acc[0][r], acc[1][r], acc[2][r], acc[3][r]};
      *reinterpret_cast<f4*>(dst) = v;
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (d + c < D) dst[c] = acc[c][r];
    }
  }
}

template <typename TX, int MG>
struct FwdTile {
  typedef Path<TX> PT;
  static constexpr int DW = tile_channels<TX>();
  static constexpr int CPW = DW / NWAVES;     // channels per wave
  static constexpr int NGRP = CPW / 4;       // scan groups of 4 channels
  static constexpr int NSTR = 16 * MG;       // floats per chunk row of the scan buffer
  static constexpr int CSTR = 16 * NSTR + 8; // floats per channel of the scan buffer
  static constexpr int WBUF = 4 * CSTR;      // floats per wave
  static constexpr int NM = fwd_mats(MG);
  static constexpr int PAIRS = NGRP * MG;    // (group, mode group) states per scan lane
};

// S = V x for the 4 channels of a group into the wave's scan buffer.
template <typename TX, int MG>
__device__ __forceinline__ void group_states(const char* xt, float* wb, int ch0,
                                             const typename Path<TX>::AOp (&vop)[4][MG],
                                             typename Path<TX>::XOp (&xv)[4], int ln, int lq) {
  typedef FwdTile<TX, MG> F;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
  XGather<TX>::get4(xt, ch0, ln, lq, xv);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
#pragma unroll
    for (int g = 0; g < MG; ++g)
      *reinterpret_cast<f4*>(&wb[k * F::CSTR + ln * F::NSTR + g * 16 + lq * 4]) =
          Path<TX>::mma(vop[k][g], xv[k], zero);
  }
}

// ---------------------------------------------------------------------------
// Aggregate kernel: per tile and scan lane, the half-tile end states (A_0, A_1)
// from a zero start; the last tile of a row also gives the state at t = L-1
// from a zero start at its first step (alast).
// ---------------------------------------------------------------------------
template <typename TX, int MG>
__global__ __launch_bounds__(NTHREADS, MG == 1 ? 4 : 2) void fwd_agg_kernel(FwdArgs a) {
  typedef FwdTile<TX, MG> F;
  typedef typename F::PT PT;
  constexpr int DW = F::DW, CPW = F::CPW, NGRP = F::NGRP, XE = (int)sizeof(TX);
  __shared__ __align__(16) char xt[XLay<XE>::BYTES];
  __shared__ __align__(16) float sbuf[NWAVES * F::WBUF];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ln = lane & 15, lq = lane >> 4;
  const int sh = lane & 1, sm = (lane >> 1) & 7, sc = lane >> 4;
  const int nchains = (int)(a.B * a.NB);
  const int64_t tile = blockIdx.x;
  const int64_t p = tile / nchains;
  const int chain = (int)(tile % nchains);
  const int64_t b = chain / a.NB;
  const int d0 = (chain % a.NB) * DW;
  const int64_t t0 = p * TILE_T;
  const bool last = (p == a.P - 1);
  const bool full = a.fast_io && t0 + TILE_T <= a.L && d0 + DW <= a.D;
  const int cw0 = wave * CPW;
  const char* tab = reinterpret_cast<const char*>(a.tab);
  float* wb = sbuf + wave * F::WBUF;

  typename PT::AOp vop[4][MG];
  auto fetch_v = [&](int grp) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int g = 0; g < MG; ++g)
        vop[k][g] = PT::load_a(tab + (size_t)(d0 + cw0 + 4 * grp + k) * F::NM * TAB_MAT_BYTES +
                               lane * TAB_LANE_BYTES + (1 + 2 * g) * TAB_MAT_BYTES);
  };
  fetch_v(0);
  tile_load<TX>(xt, reinterpret_cast<const TX*>(a.x), b, t0, d0, a.L, a.D, full, tid);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const int nstar = (a.last_len - 1) / CHUNK, jstar = (a.last_len - 1) % CHUNK;
  float4* rec = reinterpret_cast<float4*>(a.agg) + (size_t)tile * DW * a.Mp + wave * 32 * F::PAIRS;
#pragma unroll
  for (int grp = 0; grp < NGRP; ++grp) {
    typename PT::XOp xv[4];
    group_states<TX, MG>(xt, wb, cw0 + 4 * grp, vop, xv, ln, lq);
    if (grp + 1 < NGRP) fetch_v(grp + 1);
    wave_lds_order();
    const int ch = cw0 + 4 * grp + sc;
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      const int m = g * 8 + sm;
      const float2 mu = a.scal[(size_t)(d0 + ch) * a.Mp + m].mu;
      float2 run = make_float2(0.f, 0.f), hl = run;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (8 * sh + j == nstar) hl = run;  // state entering chunk nstar (from this half's start)
        const float2 sv =
            *reinterpret_cast<const float2*>(&wb[sc * F::CSTR + (8 * sh + j) * F::NSTR + g * 16 + 2 * sm]);
        run = cfma(mu, run, sv);
      }
      const float2 oth = make_float2(swap_pair(run.x), swap_pair(run.y));
      const float2 A0 = sh ? oth : run, A1 = sh ? run : oth;
      if (sh == 0) rec[(grp * MG + g) * 32 + sc * 8 + sm] = make_float4(A0.x, A0.y, A1.x, A1.y);
      if (last && a.alast != nullptr && sh == (nstar >> 3)) {
        // state at t = L-1 from a zero start at the tile's first step
        const ModeScalars ms = a.scal[(size_t)(d0 + ch) * a.Mp + m];
        if (sh == 1) {  // half 0 contributes mu^(nstar - 8) A_0
          float2 w = A0;
          for (int i = 8; i < nstar; ++i) w = cmul(ms.mu, w);
          hl = make_float2(hl.x + w.x, hl.y + w.y);
        }
        for (int i = 0; i <= jstar; ++i) {
          const TX xv1 = *reinterpret_cast<const TX*>(xt + XLay<XE>::off(nstar * CHUNK + i) + ch * XE);
          hl = cfma(ms.lam, hl, make_float2(to_f32(xv1), 0.f));
        }
        a.alast[((size_t)b * a.Dp + d0 + ch) * a.Mp + m] = hl;
      }
    }
    wave_lds_order();
  }
}

// ---------------------------------------------------------------------------
// Carry kernel: for every (row, channel, mode) the states entering each tile.
// The tiles of a row are cut into at most 64 segments of 16 * 2^k tiles;
// thread (pair, segment) folds its segment's aggregates from zero (float64), the
// segment entry states follow from the segment aggregates in order, and each
// thread replays its segment to write the entry states of both tile halves
// (c, mu^8 c + A_0).  The last
// segment also writes the state at t = L-1: lambda^last_len c_last + alast.
// The fold order is fixed by P alone, so the result is bitwise reproducible.
// ---------------------------------------------------------------------------
constexpr int CARRY_SEG_MAX = 64;  // segments per row (threads per pair)
constexpr int CARRY_BLOCK = 16;    // records loaded together

__global__ __launch_bounds__(256) void fwd_carry_kernel(FwdArgs a, int seg_len, int nseg, int nsegp,
                                                        int pairs_per_tile, int cpw, int pairs_w) {
  __shared__ double2 sg[256];  // segment aggregates, then entry states
  const int tid = threadIdx.x;
  const int pw = 256 / nsegp;                    // pairs per block
  const int seg = tid / pw, pl = tid % pw;
  const int64_t pair = (int64_t)blockIdx.x * pw + pl;  // (chain, q)
  const int nchains = (int)(a.B * a.NB);
  const bool valid = pair < (int64_t)nchains * pairs_per_tile && seg < nseg;
  const int chain = (int)(pair / pairs_per_tile), q = (int)(pair % pairs_per_tile);
  // slot q -> (channel, mode): q = wave * 32 PAIRS + 32 (grp MG + g) + 8 c + m
  const int MG = a.Mp / 8;
  const int wv = q / (32 * pairs_w), s = q % (32 * pairs_w);
  const int grp = s / (32 * MG), g = (s / 32) % MG, c = (s / 8) % 4, m8 = s % 8;
  const int ch = wv * cpw + 4 * grp + c, m = g * 8 + m8;
  const int64_t b = chain / a.NB;
  const int d = (chain % a.NB) * (cpw * NWAVES) + ch;
  const float4* agg = reinterpret_cast<const float4*>(a.agg);
  float4* car = reinterpret_cast<float4*>(a.car);

  double2 lamT = make_double2(0.0, 0.0), mu8 = lamT;
  if (valid) {
    const ModeCarry cc = a.cc[(size_t)d * a.Mp + m];
    lamT = cc.lamT;
    mu8 = cc.mu8;
  }
  const int64_t p0 = (int64_t)seg * seg_len;
  const int nsub = seg_len / CARRY_BLOCK;
  // records of tile p0 + i of this (row, pair): base[i * stride]
  const size_t stride = (size_t)nchains * pairs_per_tile;
  const float4* base = agg + (size_t)(p0 * nchains + chain) * pairs_per_tile + q;
  float4* cbase = car + (size_t)(p0 * nchains + chain) * pairs_per_tile + q;
  const int64_t nloc = valid ? (a.P - p0 < seg_len ? a.P - p0 : seg_len) : 0;  // tiles of this segment
  float4 rec[CARRY_BLOCK];
  // pass 1: the segment's end state from zero over its tiles before the row's last
  double2 acc = make_double2(0.0, 0.0);
  for (int sb = 0; sb < nsub; ++sb) {
#pragma unroll
    for (int i = 0; i < CARRY_BLOCK; ++i) {
      const int64_t li = (int64_t)sb * CARRY_BLOCK + i;
      rec[i] = li < nloc ? base[li * stride] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int i = 0; i < CARRY_BLOCK; ++i)
      if (p0 + (int64_t)sb * CARRY_BLOCK + i < a.P - 1)
        acc = zfma(lamT, acc, zfma(mu8, make_double2(rec[i].x, rec[i].y), make_double2(rec[i].z, rec[i].w)));
  }
  sg[tid] = acc;
  __syncthreads();
  // entry state of this segment: h0, then hop over the earlier segments in order
  double2 lamS = lamT;  // lambda^(256 seg_len), seg_len a power of two
  for (int e = seg_len; e > 1; e >>= 1) lamS = zmul(lamS, lamS);
  double2 ent = make_double2(0.0, 0.0);
  if (valid && a.h0 != nullptr && d < a.D && m < a.M) {
    const float* h = a.h0 + ((size_t)(b * a.D + d) * a.M + m) * 2;
    ent = make_double2(h[0], h[1]);
  }
  for (int s2 = 0; s2 < seg; ++s2) ent = zfma(lamS, ent, sg[s2 * pw + pl]);
  if (!valid) return;
  // pass 2: replay, writing the entry states of every tile of the segment
  double2 cst = ent;
  for (int sb = 0; sb < nsub; ++sb) {
    if (nsub > 1) {  // a single block is still in registers
#pragma unroll
      for (int i = 0; i < CARRY_BLOCK; ++i) {
        const int64_t li = (int64_t)sb * CARRY_BLOCK + i;
        rec[i] = li < nloc ? base[li * stride] : make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int i = 0; i < CARRY_BLOCK; ++i) {
      const int64_t li = (int64_t)sb * CARRY_BLOCK + i;
      if (li < nloc) {
        const double2 A0 = make_double2(rec[i].x, rec[i].y), A1 = make_double2(rec[i].z, rec[i].w);
        const double2 half = zfma(mu8, cst, A0);
        if (car != nullptr)
          cbase[li * stride] = make_float4((float)cst.x, (float)cst.y, (float)half.x, (float)half.y);
        if (p0 + li == a.P - 1) {
          if (a.h_out != nullptr && d < a.D && m < a.M) {
            const double2 lE = a.cc[(size_t)d * a.Mp + m].lamEll;
            const float2 al = a.alast[((size_t)b * a.Dp + d) * a.Mp + m];
            const double2 hL = zfma(lE, cst, make_double2(al.x, al.y));
            float* ho = a.h_out + ((size_t)(b * a.D + d) * a.M + m) * 2;
            ho[0] = (float)hL.x;
            ho[1] = (float)hL.y;
          }
        } else {
          cst = zfma(lamT, cst, zfma(mu8, A0, A1));
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Apply kernel: each scan lane runs its 8 chunks from its half's entry state
// and leaves the state entering every chunk in the scan buffer; then per channel
// y = T x + U H on MFMA, written over the drive column; the tile leaves as rows.
// ---------------------------------------------------------------------------
template <typename TX, typename TY, int MG>
__global__ __launch_bounds__(NTHREADS, MG == 1 ? 4 : 2) void fwd_apply_kernel(FwdArgs a) {
  typedef FwdTile<TX, MG> F;
  typedef typename F::PT PT;
  constexpr int DW = F::DW, CPW = F::CPW, NGRP = F::NGRP;
  // bf16 drive with float32 output: y leaves straight from the MFMA registers
  constexpr bool SEPY = !__is_same(TX, TY);
  __shared__ __align__(16) char xt[XLay<sizeof(TX)>::BYTES];
  __shared__ __align__(16) float sbuf[NWAVES * F::WBUF];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ln = lane & 15, lq = lane >> 4;
  const int sh = lane & 1, sm = (lane >> 1) & 7, sc = lane >> 4;
  const int nchains = (int)(a.B * a.NB);
  const int64_t tile = blockIdx.x;
  const int64_t p = tile / nchains;
  const int chain = (int)(tile % nchains);
  const int64_t b = chain / a.NB;
  const int d0 = (chain % a.NB) * DW;
  const int64_t t0 = p * TILE_T;
  const bool full = a.fast_io && t0 + TILE_T <= a.L && d0 + DW <= a.D;
  const int cw0 = wave * CPW;
  const char* tab = reinterpret_cast<const char*>(a.tab);
  float* wb = sbuf + wave * F::WBUF;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};

  auto tab_of = [&](int ch) {
    return tab + (size_t)(d0 + ch) * F::NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
  };
  typedef StateRow SO;
  typename PT::AOp vop[4][MG], top[4];
  f4 uop[4][MG];
  auto fetch_v = [&](int grp) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
      for (int g = 0; g < MG; ++g) vop[k][g] = PT::load_a(tab_of(cw0 + 4 * grp + k) + (1 + 2 * g) * TAB_MAT_BYTES);
  };
  auto fetch_tu = [&](int grp) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const char* tp = tab_of(cw0 + 4 * grp + k);
      top[k] = PT::load_a(tp);
#pragma unroll
      for (int g = 0; g < MG; ++g) uop[k][g] = load_f4(tp + (2 + 2 * g) * TAB_MAT_BYTES);
    }
  };
  // entry state of this lane's half, per (group, mode group)
  const float2* car = reinterpret_cast<const float2*>(reinterpret_cast<const float4*>(a.car) +
                                                      (size_t)tile * DW * a.Mp + wave * 32 * F::PAIRS);
  float2 ent[NGRP][MG];
#pragma unroll
  for (int grp = 0; grp < NGRP; ++grp)
#pragma unroll
    for (int g = 0; g < MG; ++g) ent[grp][g] = car[2 * ((grp * MG + g) * 32 + sc * 8 + sm) + sh];
  fetch_v(0);
  fetch_tu(0);
  tile_load<TX>(xt, reinterpret_cast<const TX*>(a.x), b, t0, d0, a.L, a.D, full, tid);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

#pragma unroll
  for (int grp = 0; grp < NGRP; ++grp) {
    typename PT::XOp xv[4];
    group_states<TX, MG>(xt, wb, cw0 + 4 * grp, vop, xv, ln, lq);
    if (grp + 1 < NGRP) fetch_v(grp + 1);
    wave_lds_order();
#pragma unroll
    for (int g = 0; g < MG; ++g) {
      const float2 mu = a.scal[(size_t)(d0 + cw0 + 4 * grp + sc) * a.Mp + g * 8 + sm].mu;
      float2 run = ent[grp][g];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float* row = &wb[sc * F::CSTR + (8 * sh + j) * F::NSTR + g * 16];
        const float2 sv = *reinterpret_cast<const float2*>(row + 2 * sm);
        SO::put(row, sm, run);  // state entering chunk 8 sh + j
        run = cfma(mu, run, sv);
      }
    }
    wave_lds_order();
    f4 acc[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      acc[k] = PT::mma(top[k], xv[k], zero);
#pragma unroll
      for (int g = 0; g < MG; ++g)
        acc[k] = SO::apply(uop[k][g], &wb[k * F::CSTR + ln * F::NSTR + g * 16], lq, acc[k]);
    }
    if (SEPY)
      put_y4_global(reinterpret_cast<float*>(a.y), acc, b, t0 + ln * CHUNK + lq * 4, d0 + cw0 + 4 * grp,
                    a.L, a.D);
    else
      put_y4<TY>(xt, cw0 + 4 * grp, ln, lq, acc);
    if (grp + 1 < NGRP) fetch_tu(grp + 1);
    wave_lds_order();
  }
  if (!SEPY) {
    __syncthreads();
    tile_store<TY>(reinterpret_cast<TY*>(a.y), xt, b, t0, d0, a.L, a.D, full, tid);
  }
}

// ---------------------------------------------------------------------------
// Single-kernel forward over row segments (one mode group, M <= 8).
//
// A work-group (8 waves) owns seg_len consecutive tiles of one chain (batch row
// b, channel block); each wave owns CW channels of the tile and keeps their
// operands in registers for the whole segment.  Per channel the state MFMA
// S = V x leaves, in lane (n, q), the drives of chunk n for the modes 2q and
// 2q+1; everything on the chunk axis then runs across the 16 lanes of a row.
//   pass 1  per tile, lane-wise acc = lambda^256 acc + mu^(15-n) S; the row sum
//           of acc is the segment's own end state from a zero start (agg_s);
//   carry   per wave (its channels form their own sub-chain): publish agg_s,
//           wait for the aggregates of all earlier segments of the row and
//           fold them, with the row's initial state, into the state entering
//           the segment (a fixed-order weighted sum, lanes in parallel);
//   pass 2  the segment streams again: per tile and channel, the entering state
//           c is added to lane 0 as mu c, the chunk recurrence
//           Q[n] = mu Q[n-1] + S[n] is a four-step prefix scan over the row
//           (shifts 1, 2, 4, 8 with multipliers mu, mu^2, mu^4, mu^8), the
//           state entering chunk n is Q[n-1] (c for n = 0) and feeds
//           y = T x + U H directly as the float32 MFMA operand; Q[15] is the
//           next tile's entering state.
// Tiles stream through three LDS tile buffers; wave 0 alone issues the
// direct-to-LDS loads (two tiles in flight), the other waves store the output
// rows.  Work-groups take segments in ticket order (time-major over the chains),
// so every wait is on a smaller ticket, which a running work-group took and
// publishes without waiting; every wait is bounded.  Payloads and flags are agent-coherent (device-scope)
// accesses; a publisher completes its payload stores before the flag store.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void st_agent(float2* p, float2 v) {
  __hip_atomic_store(reinterpret_cast<uint64_t*>(p), __builtin_bit_cast(uint64_t, v),
                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_agent(const float2* p) {
  return __builtin_bit_cast(float2, __hip_atomic_load(reinterpret_cast<const uint64_t*>(p),
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}
// the two modes of a lane as (re, im, re, im)
__device__ __forceinline__ void st_agent4(float2* p, f4 v) {
  st_agent(p, make_float2(v[0], v[1]));
  st_agent(p + 1, make_float2(v[2], v[3]));
}
__device__ __forceinline__ f4 ld_agent4(const float2* p) {
  const float2 u = ld_agent(p), w = ld_agent(p + 1);
  const f4 r = {u.x, u.y, w.x, w.y};
  return r;
}
__device__ __forceinline__ uint32_t ld_flag(const uint32_t* f) {
  return __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_flag(uint32_t* f, uint32_t v) {
  __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Upper bound on window polls (about a second); reached only if a predecessor
// never publishes, which the ticket order rules out.  The wave then starts from
// the row's initial state and records the event in the error word.
constexpr uint32_t SPIN_LIMIT = 1u << 20;

// Complex arithmetic on the two modes of a lane, (re_a, im_a, re_b, im_b).
__device__ __forceinline__ f4 c2mul(const f4& a, const f4& b) {
  f4 r;
  r[0] = fmaf(a[0], b[0], -a[1] * b[1]);
  r[1] = fmaf(a[0], b[1], a[1] * b[0]);
  r[2] = fmaf(a[2], b[2], -a[3] * b[3]);
  r[3] = fmaf(a[2], b[3], a[3] * b[2]);
  return r;
}
__device__ __forceinline__ f4 c2fma(const f4& a, const f4& b, const f4& c) {  // a b + c
  f4 r;
  r[0] = fmaf(a[0], b[0], fmaf(-a[1], b[1], c[0]));
  r[1] = fmaf(a[0], b[1], fmaf(a[1], b[0], c[1]));
  r[2] = fmaf(a[2], b[2], fmaf(-a[3], b[3], c[2]));
  r[3] = fmaf(a[2], b[3], fmaf(a[3], b[2], c[3]));
  return r;
}
__device__ __forceinline__ f4 mode_pair(float2 u, float2 w) {
  const f4 r = {u.x, u.y, w.x, w.y};
  return r;
}

// Lane moves inside rows of 16 lanes (DPP).  BOUND0: lanes without a source
// lane read zero; otherwise they keep `old`.
constexpr int DPP_ROW_SHL(int n) { return 0x100 + n; }   // lane i <- lane i + n
constexpr int DPP_ROW_SHR(int n) { return 0x110 + n; }   // lane i <- lane i - n
constexpr int DPP_QUAD(int a, int b, int c, int d) { return a | (b << 2) | (c << 4) | (d << 6); }
constexpr int DPP_ROW_MIRROR = 0x140;                    // lane i <- lane 15 - i
constexpr int DPP_ROW_HALF_MIRROR = 0x141;               // lane i <- lane 7 - i (per half row)
template <int CTRL, bool BOUND0>
__device__ __forceinline__ f4 dpp4(const f4& old, const f4& v) {
  f4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float o = old[i], x = v[i];  // scalars: a vector element is no lvalue for bit_cast
    r[i] = __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, o),
                                                                 __builtin_bit_cast(int, x), CTRL,
                                                                 0xF, 0xF, BOUND0));
  }
  return r;
}
// Sum over the 16 lanes of each row, in every lane of the row (the same order in
// every lane, so the copies agree bitwise).
__device__ __forceinline__ f4 row_sum(f4 v) {
  v += dpp4<DPP_QUAD(1, 0, 3, 2), false>(v, v);
  v += dpp4<DPP_QUAD(2, 3, 0, 1), false>(v, v);
  v += dpp4<DPP_ROW_HALF_MIRROR, false>(v, v);
  v += dpp4<DPP_ROW_MIRROR, false>(v, v);
  return v;
}

template <typename TX>
struct SegGeo {
  static constexpr int DW = tile_channels<TX>();
  static constexpr int NW = SEG_WAVES;  // waves
  static constexpr int CW = DW / NW;    // channels per wave (bf16 8, float 4)
  static constexpr int NG = CW / 4;     // operand gathers of 4 channels per wave
  static constexpr int NT = 64 * NW;    // threads
  static constexpr int NBUF = 3;        // LDS tile buffers (two loads in flight)
};

// s_waitcnt until at most n vector-memory operations of this wave are
// outstanding (expcnt and lgkmcnt not waited on); n < 64.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Drive tile into one LDS buffer (all threads call).  Full tiles: wave 0 alone
// issues the direct-to-LDS loads, so the loads are the only vector-memory
// operations it has in flight and it can wait for them exactly; other tiles:
// element loads by all threads, zeros outside the tensor.
template <typename TX>
__device__ __forceinline__ void seg_tile_load(char* xt, const TX* x, int64_t b, int64_t t0, int d0,
                                              int64_t L, int D, bool full, int tid, int wave) {
  typedef SegGeo<TX> G;
  constexpr int DW = G::DW, XE = (int)sizeof(TX);
  const int lane = tid & 63;
  if (full) {
    if (wave == 0) {
      const char* src = reinterpret_cast<const char*>(x) + ((b * L + t0) * D + d0) * XE;
      const int64_t rowb = (int64_t)D * XE;
      const uint32_t loff = (uint32_t)((lane >> 3) * rowb) + (lane & 7) * 16;  // per-lane part
#pragma unroll
      for (int g = 0; g < TILE_T / 8; ++g)
        __builtin_amdgcn_global_load_lds((gvoid_t*)(src + (int64_t)(8 * g) * rowb + loff),
                                         (lvoid_t*)(xt + g * XLay<XE>::GRP), 16, 0, 0);
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += G::NT) {
      const int t = idx / DW, c = idx % DW;
      TX v = from_f32<TX>(0.f);
      if (t0 + t < L && d0 + c < D) v = x[(b * L + t0 + t) * (int64_t)D + d0 + c];
      *reinterpret_cast<TX*>(xt + XLay<XE>::off(t) + c * XE) = v;
    }
  }
}

// Output tile from one LDS buffer (all threads call).  Full tiles: 16-byte row
// stores by waves 1 .. NW-1 (wave 0 keeps a load-only queue); other tiles:
// guarded element stores by all threads.
template <typename TY>
__device__ __forceinline__ void seg_tile_store(TY* y, const char* xt, int64_t b, int64_t t0, int d0,
                                               int64_t L, int D, bool full, int tid, int wave) {
  typedef SegGeo<TY> G;
  constexpr int DW = G::DW, YE = (int)sizeof(TY);
  const int lane = tid & 63;
  if (full) {
    if (wave > 0) {
      char* dst = reinterpret_cast<char*>(y) + ((b * L + t0) * D + d0) * YE;
      const int64_t rowb = (int64_t)D * YE;
      const uint32_t loff = (uint32_t)((lane >> 3) * rowb) + (lane & 7) * 16;  // per-lane part
      for (int g = wave - 1; g < TILE_T / 8; g += G::NW - 1) {
        const uint4 v = *reinterpret_cast<const uint4*>(xt + g * XLay<YE>::GRP + lane * 16);
        *reinterpret_cast<uint4*>(dst + (int64_t)(8 * g) * rowb + loff) = v;
      }
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += G::NT) {
      const int t = idx / DW, c = idx % DW;
      if (t0 + t < L && d0 + c < D)
        y[(b * L + t0 + t) * (int64_t)D + d0 + c] = *reinterpret_cast<const TY*>(xt + XLay<YE>::off(t) + c * YE);
    }
  }
}

template <typename TX, typename TY>
__global__ __launch_bounds__(SegGeo<TX>::NT, 1) void fwd_seg_kernel(FwdArgs a) {
  typedef SegGeo<TX> G;
  typedef Path<TX> PT;
  constexpr int DW = G::DW, NW = G::NW, CW = G::CW, NG = G::NG, XE = (int)sizeof(TX);
  constexpr int NM = fwd_mats(1);  // T, V, U
  // bf16 drive with float32 output: y leaves straight from the MFMA registers
  constexpr bool SEPY = !__is_same(TX, TY);
  __shared__ __align__(16) char xb[G::NBUF][XLay<XE>::BYTES];
  // per (channel, power s, row q): mu^(2^s) of the modes 2q, 2q+1
  __shared__ __align__(16) f4 s_pw[DW * 4 * 4];
  // per (channel, row q): the state entering the next tile; then a zero entry
  __shared__ __align__(16) f4 s_c[DW * 4 + 1];
  __shared__ uint32_t s_tk;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int ln = lane & 15, lq = lane >> 4;                   // chunk, mode pair (2 lq, 2 lq + 1)
  const int nchains = (int)(a.B * a.NB);
  const f4 zero = {0.f, 0.f, 0.f, 0.f};

  if (tid == 0) s_tk = atomicAdd(a.ticket, 1u);
  __syncthreads();
  const int64_t tk = (int64_t)__builtin_amdgcn_readfirstlane(s_tk);
  const int64_t seg = tk / nchains;
  const int chain = (int)(tk % nchains);
  const int64_t b = chain / a.NB;
  const int d0 = (chain % a.NB) * DW;
  const int64_t pb = seg * a.seg_len;                                 // first tile
  const int nt = (int)(a.P - pb < a.seg_len ? a.P - pb : a.seg_len);  // tiles of the segment
  const bool last_seg = (seg == a.seg_per_chain - 1);
  const int c0 = wave * CW;  // this wave's first channel within the tile

  const char* tab = reinterpret_cast<const char*>(a.tab);
  auto tab_of = [&](int k) {
    return tab + (size_t)(d0 + c0 + k) * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
  };
  // scalars of the lane's two modes of channel c0 + k
  auto scal_of = [&](int k) { return a.scal + (size_t)(d0 + c0 + k) * a.Mp + 2 * lq; };

  auto tile_full = [&](int64_t p) {
    return a.fast_io && (p + 1) * TILE_T <= a.L && d0 + DW <= a.D;
  };
  auto load = [&](int i) {
    const int64_t p = pb + i;
    seg_tile_load<TX>(xb[i % G::NBUF], reinterpret_cast<const TX*>(a.x), b, p * TILE_T, d0, a.L, a.D,
                      tile_full(p), tid, wave);
  };
  // wave 0 issues the tile loads and no stores: wait until tile i's loads are in
  // while tile i+1's (issued later, if by direct-to-LDS loads) stay in flight.
  // (Loads complete in order among themselves; with float32 outputs stored
  // straight from registers wave 0 also stores, so it then waits for all.)
  auto wait_tile = [&](int i) {
    if (wave == 0) {
      if (!SEPY && i + 1 < nt && tile_full(pb + i + 1))
        wait_vmcnt<TILE_T / 8>();
      else
        __builtin_amdgcn_s_waitcnt(0);
    }
  };

  typename PT::AOp vop[CW];
#pragma unroll
  for (int k = 0; k < CW; ++k) vop[k] = PT::load_a(tab_of(k) + TAB_MAT_BYTES);
  // scan multipliers mu, mu^2, mu^4, mu^8 = lambda^(16 j), j = 1, 2, 4, 8
  for (int e = tid; e < DW * 4 * MODES_PER_GROUP; e += G::NT) {
    const int ch = e / (4 * MODES_PER_GROUP), sp = (e / MODES_PER_GROUP) % 4, m = e % MODES_PER_GROUP;
    reinterpret_cast<float2*>(s_pw)[e] = a.mpow[((size_t)(d0 + ch) * CHUNK + (1 << sp)) * a.Mp + m];
  }
  if (tid < 4) s_c[DW * 4][tid] = 0.f;

  // ---- pass 1: the segment's own end state ---------------------------------
  f4 sagg[CW];
  {
    f4 w[CW], lt[CW];
#pragma unroll
    for (int k = 0; k < CW; ++k) {
      // mu^(15-n) of the lane's modes (rows [d][j][Mp] of lambda^(16 j))
      w[k] = load_f4(a.mpow + ((size_t)(d0 + c0 + k) * CHUNK + (CHUNK - 1 - ln)) * a.Mp + 2 * lq);
      const ModeScalars* ms = scal_of(k);
      lt[k] = mode_pair(ms[0].lamT, ms[1].lamT);
      sagg[k] = zero;
    }
    load(0);
    if (nt > 1) load(1);
    for (int i = 0; i < nt; ++i) {
      wait_tile(i);
      __syncthreads();  // tile i is in; every wave is done with tile i-1's buffer
      if (i + 2 < nt) load(i + 2);
      const char* xt = xb[i % G::NBUF];
#pragma unroll
      for (int gr = 0; gr < NG; ++gr) {
        typename PT::XOp xv[4];
        XGather<TX>::get4(xt, c0 + 4 * gr, ln, lq, xv);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const int k = 4 * gr + kk;
          sagg[k] = c2fma(lt[k], sagg[k], c2mul(w[k], PT::mma(vop[k], xv[kk], zero)));
        }
      }
    }
  }
#pragma unroll
  for (int k = 0; k < CW; ++k) sagg[k] = row_sum(sagg[k]);

  // ---- the state entering the segment (per wave sub-chain) ----------------------
  // c = lamS^seg h0 + sum_{j<seg} lamS^(seg-1-j) agg_j with lamS = lambda^(256
  // seg_len): term u = seg-1-j (u = seg: h0) goes to lane u % 16 of every row,
  // weighted by lamS^(u % 16) and summed over the row; blocks of 16 terms are
  // combined farthest first by Horner's rule with lamS^16.  The order is fixed
  // by seg alone, so the result is bitwise reproducible.
  const int64_t sub = tk * NW + wave;
  // payload of sub-chain s, channel k: 8 modes as float2; the lane's pair at 2 lq
  auto pay = [&](int64_t s, int k) { return ((size_t)s * CW + k) * MODES_PER_GROUP + 2 * lq; };
  if (!last_seg) {  // publish this segment's own end state
    if (ln == 0)
#pragma unroll
      for (int k = 0; k < CW; ++k) st_agent4(a.pay_agg + pay(sub, k), sagg[k]);
    __builtin_amdgcn_s_waitcnt(0);
    if (lane == 0) st_flag(a.flags + sub, FLAG_AGG);
  }
  // wait until every earlier segment of the row has published
  for (int64_t top = seg - 1; top >= 0; top -= 64) {
    const int64_t j = top - lane;
    for (uint32_t it = 0;; ++it) {
      const bool ok = j < 0 || ld_flag(a.flags + (j * nchains + chain) * NW + wave) != FLAG_NONE;
      if (__ballot(!ok) == 0) break;
      if (it >= SPIN_LIMIT) {
        if (lane == 0) atomicOr(a.error, 1u);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  f4 carry[CW];
  {
    // lamS^n of the lane's modes (rows [d][n][Mp], n = 0..16)
    auto spw = [&](int k, int n) {
      return load_f4(a.spow + ((size_t)(d0 + c0 + k) * (CHUNK + 1) + n) * a.Mp + 2 * lq);
    };
    f4 wn[CW], w16[CW];
#pragma unroll
    for (int k = 0; k < CW; ++k) {
      wn[k] = spw(k, ln);
      w16[k] = spw(k, CHUNK);
      carry[k] = zero;
    }
    for (int64_t blk = seg / CHUNK; blk >= 0; --blk) {
      const int64_t u = blk * CHUNK + ln;
      f4 v[CW];
#pragma unroll
      for (int k = 0; k < CW; ++k) {
        v[k] = zero;
        if (u < seg) {
          v[k] = ld_agent4(a.pay_agg + pay(((seg - 1 - u) * nchains + chain) * NW + wave, k));
        } else if (u == seg && a.h0 != nullptr && d0 + c0 + k < a.D) {
          const float* h = a.h0 + ((size_t)(b * a.D + d0 + c0 + k) * a.M + 2 * lq) * 2;
          if (2 * lq < a.M) v[k][0] = h[0], v[k][1] = h[1];
          if (2 * lq + 1 < a.M) v[k][2] = h[2], v[k][3] = h[3];
        }
      }
#pragma unroll
      for (int k = 0; k < CW; ++k) carry[k] = c2fma(w16[k], carry[k], row_sum(c2mul(wn[k], v[k])));
    }
  }

  // ---- pass 2: the chunk scans and the outputs ----------------------------------
  const int nstar = (a.last_len - 1) / CHUNK, jstar = (a.last_len - 1) % CHUNK;
  __syncthreads();  // every wave is done with pass 1's buffers
  load(0);
  if (nt > 1) load(1);
  typename PT::AOp top[CW];
  f4 uop[CW];
#pragma unroll
  for (int k = 0; k < CW; ++k) {
    top[k] = PT::load_a(tab_of(k));
    uop[k] = load_f4(tab_of(k) + 2 * TAB_MAT_BYTES);
    if (ln == 0) s_c[(c0 + k) * 4 + lq] = carry[k];
  }
  wave_lds_order();
  for (int i = 0; i < nt; ++i) {
    wait_tile(i);
    __syncthreads();  // tile i is in; every wave is done with tile i-1's buffer
    if (i + 2 < nt) load(i + 2);
    char* xt = xb[i % G::NBUF];
    const int64_t p = pb + i;
#pragma unroll
    for (int gr = 0; gr < NG; ++gr) {
      typename PT::XOp xv[4];
      XGather<TX>::get4(xt, c0 + 4 * gr, ln, lq, xv);
      f4 acc[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int k = 4 * gr + kk;
        const f4* pw = s_pw + (c0 + k) * 16 + lq;  // mu^(2^s) at pw[4 s]
        // the entering state c in lane 0 of each row, zero in the others
        const f4 c = s_c[ln == 0 ? (c0 + k) * 4 + lq : DW * 4];
        // Q[n] = sum_{j <= n} mu^(n-j) S[j] + mu^(n+1) c, four shift steps
        f4 q = c2fma(pw[0], c, PT::mma(vop[k], xv[kk], zero));
        q = c2fma(pw[0], dpp4<DPP_ROW_SHR(1), true>(zero, q), q);
        q = c2fma(pw[4], dpp4<DPP_ROW_SHR(2), true>(zero, q), q);
        q = c2fma(pw[8], dpp4<DPP_ROW_SHR(4), true>(zero, q), q);
        q = c2fma(pw[12], dpp4<DPP_ROW_SHR(8), true>(zero, q), q);
        const f4 h = dpp4<DPP_ROW_SHR(1), false>(c, q);  // state entering chunk n (c for n = 0)
        if (ln == CHUNK - 1) s_c[(c0 + k) * 4 + lq] = q;   // state after the tile
        acc[kk] = mma_f32(uop[k], h, PT::mma(top[k], xv[kk], zero));
        if (p == a.P - 1 && a.h_out != nullptr && ln == nstar) {
          // terminal state at t = L-1 from the state entering chunk nstar
          const int d = d0 + c0 + k;
          const ModeScalars* ms = scal_of(k);
          const f4 lam = mode_pair(ms[0].lam, ms[1].lam);
          f4 hl = h;
          for (int j = 0; j <= jstar; ++j) {
            const float xr = to_f32(*reinterpret_cast<const TX*>(xt + XLay<XE>::off(nstar * CHUNK + j) +
                                                                 (c0 + k) * XE));
            const f4 xin = {xr, 0.f, xr, 0.f};
            hl = c2fma(lam, hl, xin);
          }
          if (d < a.D) {
            float* ho = a.h_out + ((size_t)(b * a.D + d) * a.M + 2 * lq) * 2;
            if (2 * lq < a.M) ho[0] = hl[0], ho[1] = hl[1];
            if (2 * lq + 1 < a.M) ho[2] = hl[2], ho[3] = hl[3];
          }
          wave_lds_order();  // the drive reads above precede the output writes below
        }
      }
      if (SEPY)
        put_y4_global(reinterpret_cast<float*>(a.y), acc, b, p * TILE_T + ln * CHUNK + lq * 4,
                      d0 + c0 + 4 * gr, a.L, a.D);
      else
        put_y4<TY>(xt, c0 + 4 * gr, ln, lq, acc);
    }
    if (!SEPY) {
      __syncthreads();  // the whole output tile is in the buffer
      seg_tile_store<TY>(reinterpret_cast<TY*>(a.y), xt, b, p * TILE_T, d0, a.L, a.D, tile_full(p), tid,
                         wave);
    }
  }
}

__global__ void fill_zero_kernel(float* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

// ---------------------------------------------------------------------------
// Host-side launchers
// ---------------------------------------------------------------------------
template <typename TA>
hipError_t launch_prep(const Geometry& g, const float* gamma, const float* omega, const float* amp,
                       const float* phase, bool bwd, void* tab, ModeScalars* scal, ModeCarry* cc,
                       hipStream_t st, float2* mpow, float2* spow, uint32_t* flags, int64_t nflags) {
  if (bwd)
    hipLaunchKernelGGL((prep_kernel<TA, true>), dim3(g.Dp), dim3(256), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, g.seg_len * TILE_T, (TA*)tab, scal, cc, mpow,
                       spow, flags, nflags);
  else
    hipLaunchKernelGGL((prep_kernel<TA, false>), dim3(g.Dp), dim3(256), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, g.seg_len * TILE_T, (TA*)tab, scal, cc, mpow,
                       spow, flags, nflags);
  return hipGetLastError();
}
template hipError_t launch_prep<float>(const Geometry&, const float*, const float*, const float*,
                                       const float*, bool, void*, ModeScalars*, ModeCarry*,
                                       hipStream_t, float2*, float2*, uint32_t*, int64_t);
template hipError_t launch_prep<bf16_t>(const Geometry&, const float*, const float*, const float*,
                                        const float*, bool, void*, ModeScalars*, ModeCarry*,
                                        hipStream_t, float2*, float2*, uint32_t*, int64_t);

template <typename TX>
hipError_t launch_fwd_agg(const Geometry& g, const FwdArgs& a, hipStream_t st, hipEvent_t ev0,
                          hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.P * g.NB)), block(NTHREADS);
  if (g.MG == 1)
    launch_timed(fwd_agg_kernel<TX, 1>, grid, block, st, ev0, ev1, a);
  else
    launch_timed(fwd_agg_kernel<TX, 2>, grid, block, st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_agg<float>(const Geometry&, const FwdArgs&, hipStream_t, hipEvent_t,
                                          hipEvent_t);
template hipError_t launch_fwd_agg<bf16_t>(const Geometry&, const FwdArgs&, hipStream_t, hipEvent_t,
                                           hipEvent_t);

hipError_t launch_fwd_carry(const Geometry& g, const FwdArgs& a, hipStream_t st) {
  // segments: at most CARRY_SEG_MAX per row, CARRY_BLOCK * 2^k tiles each
  int seg_len = CARRY_BLOCK;
  while ((g.P + seg_len - 1) / seg_len > CARRY_SEG_MAX) seg_len *= 2;
  const int nseg = (int)((g.P + seg_len - 1) / seg_len);
  int nsegp = 1;
  while (nsegp < nseg) nsegp *= 2;
  const int pw = 256 / nsegp;
  const int pairs_per_tile = g.DW * g.Mp;
  const int64_t npairs = g.B * g.NB * (int64_t)pairs_per_tile;
  const int cpw = g.DW / NWAVES;
  const int pairs_w = (cpw / 4) * g.MG;
  hipLaunchKernelGGL(fwd_carry_kernel, dim3((unsigned)((npairs + pw - 1) / pw)), dim3(256), 0, st, a,
                     seg_len, nseg, nsegp, pairs_per_tile, cpw, pairs_w);
  return hipGetLastError();
}

template <typename TX, typename TY>
hipError_t launch_fwd_segments(const Geometry& g, const FwdArgs& a, hipStream_t st, hipEvent_t ev0,
                               hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.NB * a.seg_per_chain)), block(SegGeo<TX>::NT);
  launch_timed(fwd_seg_kernel<TX, TY>, grid, block, st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_segments<float, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                      hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_segments<bf16_t, bf16_t>(const Geometry&, const FwdArgs&, hipStream_t,
                                                        hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_segments<bf16_t, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                       hipEvent_t, hipEvent_t);

template <typename TX, typename TY>
hipError_t launch_fwd_apply(const Geometry& g, const FwdArgs& a, hipStream_t st, hipEvent_t ev0,
                            hipEvent_t ev1) {
  const dim3 grid((unsigned)(g.B * g.P * g.NB)), block(NTHREADS);
  if (g.MG == 1)
    launch_timed(fwd_apply_kernel<TX, TY, 1>, grid, block, st, ev0, ev1, a);
  else
    launch_timed(fwd_apply_kernel<TX, TY, 2>, grid, block, st, ev0, ev1, a);
  return hipGetLastError();
}
template hipError_t launch_fwd_apply<float, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                   hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_apply<bf16_t, bf16_t>(const Geometry&, const FwdArgs&, hipStream_t,
                                                     hipEvent_t, hipEvent_t);
template hipError_t launch_fwd_apply<bf16_t, float>(const Geometry&, const FwdArgs&, hipStream_t,
                                                    hipEvent_t, hipEvent_t);

hipError_t launch_fill_zero(float* p, int64_t n, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, p, n);
  return hipGetLastError();
}

}  // namespace res
