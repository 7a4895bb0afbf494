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
                                                   uint32_t* __restrict__ flags, int64_t nflags) {
  // lambda^0..16, then lambda^128, lambda^256, lambda^last_len, lambda^seg_steps
  constexpr int NPW = CHUNK + 1 + 4;
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
                    : k == CHUNK + 3 ? last_len
                                     : seg_steps;
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
    ms.lamS = make_float2((float)pw[m][CHUNK + 4].x, (float)pw[m][CHUNK + 4].y);
    scal[(size_t)d * Mp + m] = ms;
    ModeCarry mc;
    mc.lamT = lT;
    mc.lamEll = pw[m][CHUNK + 3];
    mc.mu8 = lH;
    cc[(size_t)d * Mp + m] = mc;
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
    const bool state_mat = BWD && bwd_mat_is_state(mat);
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

constexpr int XROW = 128;                      // bytes per time row of a tile
constexpr int XGRP = 8 * XROW + 4;             // 8 rows + pad (conflict-free operand reads)
constexpr int XT_BYTES = (TILE_T / 8) * XGRP;  // 32896

__device__ __forceinline__ int xt_off(int t) { return (t >> 3) * XGRP + (t & 7) * XROW; }

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
      __builtin_amdgcn_global_load_lds((gvoid_t*)s, (lvoid_t*)(xt + g * XGRP), 16, 0, 0);
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += NTHREADS) {
      const int t = idx / DW, c = idx % DW;
      TX v = from_f32<TX>(0.f);
      if (t0 + t < L && d0 + c < D) v = x[(b * L + t0 + t) * (int64_t)D + d0 + c];
      *reinterpret_cast<TX*>(xt + xt_off(t) + c * XE) = v;
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
      const uint4 v = *reinterpret_cast<const uint4*>(xt + g * XGRP + lane * 16);
      *reinterpret_cast<uint4*>(dst + (int64_t)(8 * g + (lane >> 3)) * rowb + (lane & 7) * 16) = v;
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += NTHREADS) {
      const int t = idx / DW, c = idx % DW;
      if (t0 + t < L && d0 + c < D)
        y[(b * L + t0 + t) * (int64_t)D + d0 + c] = *reinterpret_cast<const TY*>(xt + xt_off(t) + c * YE);
    }
  }
}

// Activation operand of chunk n for channel ch from the time-major tile.
template <typename TX> struct XGather;
template <> struct XGather<bf16_t> {
  // lane (n, q): taps 8(q&1) .. +7 = rows 16n + 8(q&1) + r = group 2n + (q&1), row r
  __device__ static __forceinline__ bf8 get(const char* xt, int ch, int n, int q) {
    const char* p = xt + (2 * n + (q & 1)) * XGRP + ch * 2;
    bf8 v;
#pragma unroll
    for (int r = 0; r < 8; ++r) v[r] = *reinterpret_cast<const __bf16*>(p + r * XROW);
    return v;
  }
};
template <> struct XGather<float> {
  // lane (n, q), slot kk: tap 4q + kk = row 16n + 4q + kk = group 2n + (q>>1), row 4(q&1) + kk
  __device__ static __forceinline__ f4 get(const char* xt, int ch, int n, int q) {
    const char* p = xt + (2 * n + (q >> 1)) * XGRP + 4 * (q & 1) * XROW + ch * 4;
    f4 v;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) v[kk] = *reinterpret_cast<const float*>(p + kk * XROW);
    return v;
  }
};

__device__ __forceinline__ float swap_pair(float v) {  // value of the neighbouring lane (lane ^ 1)
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1,
                                                               0xF, 0xF, false));
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
  static constexpr int NM = 1 + 2 * MG;
  static constexpr int PAIRS = NGRP * MG;    // (group, mode group) states per scan lane
};

// S = V x for the 4 channels of a group into the wave's scan buffer.
template <typename TX, int MG>
__device__ __forceinline__ void group_states(const char* xt, float* wb, int ch0,
                                             const typename Path<TX>::AOp (&vop)[4][MG],
                                             typename Path<TX>::XOp (&xv)[4], int ln, int lq) {
  typedef FwdTile<TX, MG> F;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    xv[k] = XGather<TX>::get(xt, ch0 + k, ln, lq);
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
  __shared__ __align__(16) char xt[XT_BYTES];
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
          const TX xv1 = *reinterpret_cast<const TX*>(xt + xt_off(nstar * CHUNK + i) + ch * XE);
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
  __shared__ __align__(16) char xt[XT_BYTES];
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
  typedef StateOp<TX> SO;
  typename PT::AOp vop[4][MG], top[4];
  typename SO::UOp uop[4][MG];
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
      for (int g = 0; g < MG; ++g) uop[k][g] = SO::load_u(tp + (2 + 2 * g) * TAB_MAT_BYTES);
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
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int ch = cw0 + 4 * grp + k;
      f4 acc = PT::mma(top[k], xv[k], zero);
#pragma unroll
      for (int g = 0; g < MG; ++g)
        acc = SO::apply(uop[k][g], &wb[k * F::CSTR + ln * F::NSTR + g * 16], lq, acc);
      if (SEPY) {
        const int d = d0 + ch;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t t = t0 + ln * CHUNK + lq * 4 + r;
          if (d < a.D && t < a.L) reinterpret_cast<float*>(a.y)[(b * a.L + t) * (int64_t)a.D + d] = acc[r];
        }
      } else {
        // rows 16 ln + 4 lq + r: group 2 ln + (lq >> 1), rows 4 (lq & 1) + r
        char* dst = xt + (2 * ln + (lq >> 1)) * XGRP + 4 * (lq & 1) * XROW + ch * (int)sizeof(TY);
#pragma unroll
        for (int r = 0; r < 4; ++r) *reinterpret_cast<TY*>(dst + r * XROW) = from_f32<TY>(acc[r]);
      }
    }
    if (grp + 1 < NGRP) fetch_tu(grp + 1);
    wave_lds_order();
  }
  if (!SEPY) {
    __syncthreads();
    tile_store<TY>(reinterpret_cast<TY*>(a.y), xt, b, t0, d0, a.L, a.D, full, tid);
  }
}

// ---------------------------------------------------------------------------
// Single-kernel forward over row segments (M <= 8).
//
// A work-group owns seg_len consecutive tiles of one chain (batch row b,
// channel block) and DW/4 waves, one group of 4 channels each; a wave keeps its
// channels' T, V and U operands in registers for the whole segment.  Tiles
// stream through two LDS tile buffers: the direct-to-LDS load of the next tile
// is in flight while the current one is computed.
//   pass 1  per tile S = V x and the half folds A_0, A_1; the segment's own end
//           state agg_s = fold over its tiles of lambda^256 agg + (mu^8 A_0 + A_1)
//   look-back  per wave (its channels form their own sub-chain): publish agg_s,
//           find the state entering the segment from the nearest published
//           inclusive state and the aggregates after it (the canonical
//           recurrence inc(s) = lambda^(256 seg_len) inc(s-1) + agg_s, so the
//           result does not depend on timing), publish inc(s)
//   pass 2  the segment streams again: per tile the scan lanes run their chunks
//           from the carried state (half 1 enters with mu^8 c + A_0) leaving
//           the state entering each chunk in the scan buffer, y = T x + U H on
//           MFMA over the drive column, the tile leaves as rows; the state
//           after the tile is carried to the next tile in registers.
// Work-groups take segments in ticket order (time-major over the chains), so
// every wait is on a smaller ticket, which a running work-group took; every
// wait is bounded.  Payloads and flags are agent-coherent (device-scope)
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

template <typename TX>
struct SegGeo {
  static constexpr int DW = tile_channels<TX>();
  static constexpr int NW = SEG_WAVES;              // waves
  static constexpr int NG = DW / (4 * NW);          // scan groups of 4 channels per wave
  static constexpr int NT = 64 * NW;                // threads
  static constexpr int NSTR = 16;                   // floats per chunk row (one mode group)
  static constexpr int CSTR = 16 * NSTR + 8;        // floats per channel of the scan buffer
  static constexpr int WBUF = 4 * CSTR;             // floats per wave (one group at a time)
  static constexpr int NBUF = 3;                    // LDS tile buffers (two loads in flight)
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
                                         (lvoid_t*)(xt + g * XGRP), 16, 0, 0);
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += G::NT) {
      const int t = idx / DW, c = idx % DW;
      TX v = from_f32<TX>(0.f);
      if (t0 + t < L && d0 + c < D) v = x[(b * L + t0 + t) * (int64_t)D + d0 + c];
      *reinterpret_cast<TX*>(xt + xt_off(t) + c * XE) = v;
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
        const uint4 v = *reinterpret_cast<const uint4*>(xt + g * XGRP + lane * 16);
        *reinterpret_cast<uint4*>(dst + (int64_t)(8 * g) * rowb + loff) = v;
      }
    }
  } else {
    for (int idx = tid; idx < TILE_T * DW; idx += G::NT) {
      const int t = idx / DW, c = idx % DW;
      if (t0 + t < L && d0 + c < D)
        y[(b * L + t0 + t) * (int64_t)D + d0 + c] = *reinterpret_cast<const TY*>(xt + xt_off(t) + c * YE);
    }
  }
}

template <typename TX, typename TY>
__global__ __launch_bounds__(SegGeo<TX>::NT, 1) void fwd_seg_kernel(FwdArgs a) {
  typedef SegGeo<TX> G;
  typedef Path<TX> PT;
  typedef StateOp<TX> SO;
  constexpr int DW = G::DW, NW = G::NW, NG = G::NG, XE = (int)sizeof(TX);
  constexpr int NM = 3;  // T, V, U
  // bf16 drive with float32 output: y leaves straight from the MFMA registers
  constexpr bool SEPY = !__is_same(TX, TY);
  __shared__ __align__(16) char xb[G::NBUF][XT_BYTES];
  __shared__ __align__(16) float sbuf[NW * G::WBUF];
  __shared__ uint32_t s_tk;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);      // wave-uniform (scalar)
  const int ln = lane & 15, lq = lane >> 4;                       // MFMA layout
  const int sh = lane & 1, sm = (lane >> 1) & 7, sc = lane >> 4;  // scan layout
  const int nchains = (int)(a.B * a.NB);
  float* wb = sbuf + wave * G::WBUF;
  const f4 zero = {0.f, 0.f, 0.f, 0.f};

  if (tid == 0) s_tk = atomicAdd(a.ticket, 1u);
  __syncthreads();
  const int64_t tk = (int64_t)__builtin_amdgcn_readfirstlane(s_tk);
  const int64_t seg = tk / nchains;
  const int chain = (int)(tk % nchains);
  const int64_t b = chain / a.NB;
  const int d0 = (chain % a.NB) * DW;
  const int64_t pb = seg * a.seg_len;                               // first tile
  const int nt = (int)(a.P - pb < a.seg_len ? a.P - pb : a.seg_len);  // tiles of the segment
  const bool last_seg = (seg == a.seg_per_chain - 1);
  const int ch0 = wave * 4 * NG;  // this wave's first channel within the tile

  // resident operands T, V, U of the wave's channels
  const char* tab = reinterpret_cast<const char*>(a.tab);
  auto tab_of = [&](int k) {
    return tab + (size_t)(d0 + ch0 + k) * NM * TAB_MAT_BYTES + lane * TAB_LANE_BYTES;
  };
  typename PT::AOp top[4 * NG], vop[4 * NG];
  typename SO::UOp uop[4 * NG];
#pragma unroll
  for (int k = 0; k < 4 * NG; ++k) {
    top[k] = PT::load_a(tab_of(k));
    vop[k] = PT::load_a(tab_of(k) + TAB_MAT_BYTES);
    uop[k] = SO::load_u(tab_of(k) + 2 * TAB_MAT_BYTES);
  }
  // scan-lane scalars: group gr, channel ch0 + 4 gr + sc, mode sm
  float2 mu[NG], mu8[NG], lamT[NG];
#pragma unroll
  for (int gr = 0; gr < NG; ++gr) {
    const ModeScalars& ms = a.scal[(size_t)(d0 + ch0 + 4 * gr + sc) * a.Mp + sm];
    mu[gr] = ms.mu;
    mu8[gr] = ms.mu8;
    lamT[gr] = ms.lamT;
  }

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
  // S = V x for the 4 channels of group gr into the wave's scan buffer; keeps the operands
  auto states = [&](const char* xt, int gr, typename PT::XOp (&xv)[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      xv[k] = XGather<TX>::get(xt, ch0 + 4 * gr + k, ln, lq);
      *reinterpret_cast<f4*>(&wb[k * G::CSTR + ln * G::NSTR + lq * 4]) =
          PT::mma(vop[4 * gr + k], xv[k], zero);
    }
  };
  // row of chunk n of scan channel c (of the group in the buffer)
  auto row = [&](int c, int n) -> float* { return &wb[c * G::CSTR + n * G::NSTR]; };

  // ---- pass 1: the segment's own end state ---------------------------------
  float2 sagg[NG];
#pragma unroll
  for (int gr = 0; gr < NG; ++gr) sagg[gr] = make_float2(0.f, 0.f);
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
      states(xt, gr, xv);
      wave_lds_order();
      float2 run = make_float2(0.f, 0.f);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        run = cfma(mu[gr], run, *reinterpret_cast<const float2*>(row(sc, 8 * sh + j) + 2 * sm));
      const float2 oth = make_float2(swap_pair(run.x), swap_pair(run.y));
      const float2 A0 = sh ? oth : run, A1 = sh ? run : oth;
      sagg[gr] = cfma(lamT[gr], sagg[gr], cfma(mu8[gr], A0, A1));
      wave_lds_order();
    }
  }

  // ---- look-back over segments (per wave sub-chain) --------------------------
  const int64_t sub = tk * NW + wave;
  const int64_t stride = (int64_t)nchains * NW;  // sub-chain step between segments of a row
  auto pay = [&](int64_t s, int gr) { return ((size_t)s * NG + gr) * 32 + sc * 8 + sm; };
  float2 carry[NG];
#pragma unroll
  for (int gr = 0; gr < NG; ++gr) {
    const int d = d0 + ch0 + 4 * gr + sc;
    carry[gr] = make_float2(0.f, 0.f);
    if (a.h0 != nullptr && d < a.D && sm < a.M) {
      const float* h = a.h0 + ((size_t)(b * a.D + d) * a.M + sm) * 2;
      carry[gr] = make_float2(h[0], h[1]);
    }
  }
  if (seg > 0) {
    // publish this segment's aggregate (successors may fold it before this
    // segment's own inclusive state is released)
    if (!last_seg) {
      if (sh == 0)
#pragma unroll
        for (int gr = 0; gr < NG; ++gr) st_agent(a.pay_agg + pay(sub, gr), sagg[gr]);
      __builtin_amdgcn_s_waitcnt(0);
      if (lane == 0) st_flag(a.flags + sub, FLAG_AGG);
    }
    const uint32_t fpred = ld_flag(a.flags + sub - stride);
    int64_t jres;  // nearest segment of the row with its inclusive state out (-1: row start)
    if (fpred == FLAG_INCL) {
      jres = seg - 1;
    } else {
      int64_t top_j = seg - 1;
      jres = -2;
      uint32_t it = 0;
      while (jres == -2) {
        const int64_t j = top_j - lane;
        const uint32_t fl = (j >= 0) ? ld_flag(a.flags + (j * nchains + chain) * NW + wave) : FLAG_INCL;
        const uint64_t incl = __ballot(fl == FLAG_INCL);
        const uint64_t none = __ballot(fl == FLAG_NONE);
        if (incl != 0) {
          const int l = __ffsll((unsigned long long)incl) - 1;
          const uint64_t nearer = (l == 0) ? 0ull : (~0ull >> (64 - l));
          if ((none & nearer) == 0) jres = top_j - l;
        } else if (none == 0) {
          top_j -= 64;  // the whole window holds aggregates: keep looking further back
          continue;
        }
        if (jres == -2) {
          if (++it >= SPIN_LIMIT) {
            if (lane == 0) atomicOr(a.error, 1u);
            jres = -1;
          } else {
            __builtin_amdgcn_s_sleep(1);
          }
        }
      }
    }
    if (jres >= 0) {
      const int64_t js = (jres * nchains + chain) * NW + wave;
#pragma unroll
      for (int gr = 0; gr < NG; ++gr) carry[gr] = ld_agent(a.pay_inc + pay(js, gr));
    }
    float2 lamS[NG];
#pragma unroll
    for (int gr = 0; gr < NG; ++gr) lamS[gr] = a.scal[(size_t)(d0 + ch0 + 4 * gr + sc) * a.Mp + sm].lamS;
    constexpr int LB = 16 / NG;
    for (int64_t i = jres + 1; i < seg; i += LB) {
      const int n = (seg - i) < LB ? (int)(seg - i) : LB;
      float2 v[LB][NG];
#pragma unroll
      for (int u = 0; u < LB; ++u)
#pragma unroll
        for (int gr = 0; gr < NG; ++gr)
          v[u][gr] = (u < n) ? ld_agent(a.pay_agg + pay(((i + u) * nchains + chain) * NW + wave, gr))
                             : make_float2(0.f, 0.f);
#pragma unroll
      for (int u = 0; u < LB; ++u)
        if (u < n)
#pragma unroll
          for (int gr = 0; gr < NG; ++gr) carry[gr] = cfma(lamS[gr], carry[gr], v[u][gr]);
    }
  }
  // the inclusive state is stored now; the first segment of a row releases it
  // at once, the others once pass 2 is under way (later segments fold the
  // aggregates back to the row's first segment meanwhile)
  if (!last_seg && sh == 0)
#pragma unroll
    for (int gr = 0; gr < NG; ++gr) {
      const float2 ls = a.scal[(size_t)(d0 + ch0 + 4 * gr + sc) * a.Mp + sm].lamS;
      st_agent(a.pay_inc + pay(sub, gr), cfma(ls, carry[gr], sagg[gr]));
    }
  if (!last_seg && seg == 0) {
    __builtin_amdgcn_s_waitcnt(0);
    if (lane == 0) st_flag(a.flags + sub, FLAG_INCL);
  }

  // ---- pass 2: carried states and outputs --------------------------------------
  const int nstar = (a.last_len - 1) / CHUNK, jstar = (a.last_len - 1) % CHUNK;
  __syncthreads();  // every wave is done with pass 1's buffers
  load(0);
  if (nt > 1) load(1);
  for (int i = 0; i < nt; ++i) {
    wait_tile(i);
    if (i == 0 && !last_seg && seg > 0) {  // release the inclusive state
      __builtin_amdgcn_s_waitcnt(0);
      if (lane == 0) st_flag(a.flags + sub, FLAG_INCL);
    }
    __syncthreads();  // tile i is in; every wave is done with tile i-1's buffer
    if (i + 2 < nt) load(i + 2);
    char* xt = xb[i % G::NBUF];
    const int64_t p = pb + i;
#pragma unroll
    for (int gr = 0; gr < NG; ++gr) {
      typename PT::XOp xv[4];
      states(xt, gr, xv);
      wave_lds_order();
      // half 1 enters with mu^8 c + A_0; both halves then run their chunks
      float2 A0 = make_float2(0.f, 0.f);
      if (sh) {
#pragma unroll
        for (int j = 0; j < 8; ++j) A0 = cfma(mu[gr], A0, *reinterpret_cast<const float2*>(row(sc, j) + 2 * sm));
      }
      float2 run = sh ? cfma(mu8[gr], carry[gr], A0) : carry[gr];
      float2 hl = run;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int n = 8 * sh + j;
        const float2 sv = *reinterpret_cast<const float2*>(row(sc, n) + 2 * sm);
        SO::put(row(sc, n), sm, run);  // state entering chunk n
        if (n == nstar) hl = run;
        run = cfma(mu[gr], run, sv);
      }
      // the state after the tile (from half 1) carries to the next tile
      const float2 oth = make_float2(swap_pair(run.x), swap_pair(run.y));
      carry[gr] = sh ? run : oth;
      if (p == a.P - 1 && a.h_out != nullptr && sh == (nstar >> 3)) {
        // terminal state at t = L-1 from the state entering chunk nstar
        const int chs = ch0 + 4 * gr + sc, d = d0 + chs;
        const float2 lam = a.scal[(size_t)d * a.Mp + sm].lam;
        for (int j = 0; j <= jstar; ++j) {
          const TX xv1 = *reinterpret_cast<const TX*>(xt + xt_off(nstar * CHUNK + j) + chs * XE);
          hl = cfma(lam, hl, make_float2(to_f32(xv1), 0.f));
        }
        if (d < a.D && sm < a.M) {
          float* ho = a.h_out + ((size_t)(b * a.D + d) * a.M + sm) * 2;
          ho[0] = hl.x;
          ho[1] = hl.y;
        }
      }
      wave_lds_order();
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int ch = ch0 + 4 * gr + k;
        f4 acc = PT::mma(top[4 * gr + k], xv[k], zero);
        acc = SO::apply(uop[4 * gr + k], &wb[k * G::CSTR + ln * G::NSTR], lq, acc);
        if (SEPY) {
          const int d = d0 + ch;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int64_t t = p * TILE_T + ln * CHUNK + lq * 4 + r;
            if (d < a.D && t < a.L) reinterpret_cast<float*>(a.y)[(b * a.L + t) * (int64_t)a.D + d] = acc[r];
          }
        } else {
          // rows 16 ln + 4 lq + r: group 2 ln + (lq >> 1), rows 4 (lq & 1) + r
          char* dst = xt + (2 * ln + (lq >> 1)) * XGRP + 4 * (lq & 1) * XROW + ch * (int)sizeof(TY);
#pragma unroll
          for (int r = 0; r < 4; ++r) *reinterpret_cast<TY*>(dst + r * XROW) = from_f32<TY>(acc[r]);
        }
      }
      wave_lds_order();
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
                       hipStream_t st, uint32_t* flags, int64_t nflags) {
  if (bwd)
    hipLaunchKernelGGL((prep_kernel<TA, true>), dim3(g.Dp), dim3(256), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, g.seg_len * TILE_T, (TA*)tab, scal, cc, flags,
                       nflags);
  else
    hipLaunchKernelGGL((prep_kernel<TA, false>), dim3(g.Dp), dim3(256), 0, st, gamma, omega, amp,
                       phase, (int)g.D, (int)g.M, g.MG, g.last_len, g.seg_len * TILE_T, (TA*)tab, scal, cc, flags,
                       nflags);
  return hipGetLastError();
}
template hipError_t launch_prep<float>(const Geometry&, const float*, const float*, const float*,
                                       const float*, bool, void*, ModeScalars*, ModeCarry*,
                                       hipStream_t, uint32_t*, int64_t);
template hipError_t launch_prep<bf16_t>(const Geometry&, const float*, const float*, const float*,
                                        const float*, bool, void*, ModeScalars*, ModeCarry*,
                                       hipStream_t, uint32_t*, int64_t);

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
